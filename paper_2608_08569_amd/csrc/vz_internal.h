// Internal helpers shared by the libvoxzip kernels and the host API.
// Everything here targets gfx950 (CDNA4): wave64, 160 KB LDS per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/voxzip.h"

namespace vz {

constexpr int kWave = 64;

// ---- bfloat16 <-> float ---------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even (finite inputs; NaN becomes a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu))
        return static_cast<uint16_t>((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// Element traits: storage type, 16-byte vector width, widening.
template <int DT> struct Elem;
template <> struct Elem<VZ_F32> {
    using T = float;
    static constexpr int kPer16B = 4;
    __device__ static __forceinline__ float load(const T* p, size_t i) { return p[i]; }
    __device__ static __forceinline__ T from_f32(float f) { return f; }
    __device__ static __forceinline__ float to_f32(T x) { return x; }
};
template <> struct Elem<VZ_BF16> {
    using T = uint16_t;
    static constexpr int kPer16B = 8;
    __device__ static __forceinline__ float load(const T* p, size_t i) { return bf16_to_f32(p[i]); }
    __device__ static __forceinline__ T from_f32(float f) { return f32_to_bf16(f); }
    __device__ static __forceinline__ float to_f32(T x) { return bf16_to_f32(x); }
};

// Unpack one 16-byte vector into floats.
template <int DT>
__device__ __forceinline__ void unpack16(const uint4& v, float* out) {
    if constexpr (DT == VZ_F32) {
        out[0] = __uint_as_float(v.x); out[1] = __uint_as_float(v.y);
        out[2] = __uint_as_float(v.z); out[3] = __uint_as_float(v.w);
    } else {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            out[2 * i] = __uint_as_float(w[i] << 16);
            out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
    }
}

template <int DT>
__device__ __forceinline__ uint4 pack16(const float* in) {
    uint4 v;
    if constexpr (DT == VZ_F32) {
        v.x = __float_as_uint(in[0]); v.y = __float_as_uint(in[1]);
        v.z = __float_as_uint(in[2]); v.w = __float_as_uint(in[3]);
    } else {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = static_cast<uint32_t>(f32_to_bf16(in[2 * i])) |
                   (static_cast<uint32_t>(f32_to_bf16(in[2 * i + 1])) << 16);
        v.x = w[0]; v.y = w[1]; v.z = w[2]; v.w = w[3];
    }
    return v;
}

// ---- eviction ranking key ---------------------------------------------------
// A larger key is a more important slot: higher score first, then the smaller
// position.  The float is mapped to an order-preserving uint32 (-0 as +0).
__device__ __forceinline__ uint64_t rank_key(float score, int32_t pos) {
    uint32_t b = __float_as_uint(score);
    if (b == 0x80000000u) b = 0u;
    uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
    return (static_cast<uint64_t>(ord) << 32) | static_cast<uint64_t>(~static_cast<uint32_t>(pos));
}

// ---- wave / block reductions ------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
    uint32_t lo = static_cast<uint32_t>(v), hi = static_cast<uint32_t>(v >> 32);
    lo = __shfl_xor(lo, o, kWave);
    hi = __shfl_xor(hi, o, kWave);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        uint64_t w = shfl_xor_u64(v, o);
        v = w < v ? w : v;
    }
    return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

}  // namespace vz

// ---- launchers (one per kernel family), called by the host API -------------
struct VzDecodeArgs {
    const void* q; const void* k_new; const void* v_new;
    void* k_cache; void* v_cache; float* score; int32_t* pos; void* out;
    int32_t len, next_pos; float gamma, sm_scale;
    int32_t L, Hq, Hkv, d, cap, dtype;
    void* ws; size_t ws_bytes;
};

struct VzEvictArgs {
    void* k_cache; void* v_cache; float* score; int32_t* pos;
    int32_t len, budget, n_sink, n_recent, next_pos;
    int32_t* kept_pos_out;
    int32_t L, Hkv, d, cap, dtype;
    void* ws; size_t ws_bytes;
};

// Stage-1 span offsets (host); arguments checked by the caller; returns the
// number of spans written to off_out[1..].
int32_t vz_build_span_offsets(const int64_t* t_start_ms, const int64_t* t_end_ms, const float* conf,
                              const int32_t* text_len, int32_t n_seg, int64_t t_total_ms, int32_t L_a,
                              float conf_threshold, int32_t* off_out);
hipError_t vz_launch_fuse(const void* k_in, const void* v_in, int32_t T_in, const int32_t* off,
                          int32_t n_spans, const void* ak, const void* av, void* k_out, void* v_out,
                          float* score_out, int32_t* pos_out, int32_t L, int32_t H, int32_t d,
                          int32_t cap_out, int32_t dtype, hipStream_t stream);
size_t vz_decode_ws_bytes(int32_t L, int32_t Hq, int32_t Hkv, int32_t d, int32_t cap);
// decode workspace: a header (ticket, error flag) of vz_decode_hdr_bytes(L)
// bytes, then path-specific scratch
size_t vz_decode_hdr_bytes(int32_t L);
bool vz_decode_fused_ok(int32_t dtype, int32_t d, int32_t Hq, int32_t Hkv, int32_t cap, int32_t L);
size_t vz_decode_fused_ws_bytes(int32_t L, int32_t Hq, int32_t cap);
hipError_t vz_launch_decode_fused(const VzDecodeArgs& a, hipStream_t stream);
size_t vz_decode_generic_ws_bytes(int32_t L, int32_t Hq, int32_t cap);
hipError_t vz_launch_decode_generic(const VzDecodeArgs& a, hipStream_t stream);
hipError_t vz_launch_decode(const VzDecodeArgs& a, hipStream_t stream);
size_t vz_evict_ws_bytes(int32_t L, int32_t Hkv, int32_t d, int32_t cap);
hipError_t vz_launch_evict(const VzEvictArgs& a, hipStream_t stream);
