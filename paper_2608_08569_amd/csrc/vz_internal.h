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
// Minimum over the wave (every lane active): the high words first, then the
// low words of the lanes holding that high word; two cross-lane (DPP)
// reductions instead of six dependent 64-bit shuffles through LDS.
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
    const uint32_t hi = static_cast<uint32_t>(v >> 32), lo = static_cast<uint32_t>(v);
    const uint32_t hmin = __reduce_min_sync(~0ull, hi);
    const uint32_t lmin = __reduce_min_sync(~0ull, hi == hmin ? lo : 0xFFFFFFFFu);
    return (static_cast<uint64_t>(hmin) << 32) | lmin;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

}  // namespace vz

// ---- ragged batches ---------------------------------------------------------
// Sequence s of a ragged batch owns slots base[s] .. base[s] + cap[s] - 1 of
// every (layer, head) plane, and a plane holds `total` slots.  The
// per-sequence values are device arrays read by the kernels; a sequence whose
// values are out of range is skipped (nothing of it is read or written) and
// its status entry says why.
struct VzRagged {
    const int64_t* base;
    const int32_t* cap;
    const int32_t* len;
    const int32_t* next_pos;
    const int32_t* budget;  // eviction only
    int32_t* status;        // [n], may be null
    int32_t n;
    int64_t total;
};

// Largest plane (slots) and batch a ragged call serves: every flat chunk index
// and running count below stays far from 2^31.
constexpr int64_t kRaggedMaxTotal = int64_t(1) << 26;
constexpr int32_t kRaggedMaxSeqs = 1 << 15;  // also a grid dimension

namespace vz {

// Status of a sequence for a decode step from its values (base, cap, len,
// next_pos): VZ_OK when slot len exists and the sequence lies inside the
// planes of `total` slots, VZ_IDLE for an idle slot (cap 0).
__device__ __forceinline__ int decode_status_of(int64_t b, int c, int n, int p, int64_t total) {
    if (c == 0) return VZ_IDLE;
    if (n < 0 || p < 0 || c < 1 || b < 0 || b > total - c) return VZ_ERR_INVALID;
    if (n >= c) return VZ_ERR_CAPACITY;  // no free slot (len + 1 > cap, without overflow)
    return VZ_OK;
}
__device__ __forceinline__ int ragged_decode_status(const VzRagged& r, int s) {
    return decode_status_of(r.base[s], r.cap[s], r.len[s], r.next_pos[s], r.total);
}

// Flat work items of a ragged batch: sequence s contributes count(s) >= 0
// consecutive items, in sequence order.  Called by a whole wave (every lane
// gets the same result, wave-uniform).  Returns the sequence holding flat item
// f, with its first flat item and its item count, or -1 when f lies past
// `limit` items or past the last one.  count() must return at most 2^24.
template <class Count>
__device__ int ragged_locate(int f, int n_seqs, int limit, Count count, int& first, int& nc) {
    const int lane = threadIdx.x % kWave;
    int run = 0;
    for (int s0 = 0; s0 < n_seqs && run <= limit; s0 += kWave) {
        const int s = s0 + lane;
        const int n0 = count(s < n_seqs ? s : n_seqs - 1);  // load for every lane, mask after
        const int n = s < n_seqs ? n0 : 0;
        int incl = n;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int t = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += t;
        }
        const unsigned long long hit = __ballot(run + incl > f);
        if (hit) {
            const int src = __builtin_ctzll(hit);
            nc = __builtin_amdgcn_readfirstlane(__shfl(n, src, kWave));
            first = __builtin_amdgcn_readfirstlane(run + __shfl(incl, src, kWave) - nc);
            return __builtin_amdgcn_readfirstlane(s0 + src);
        }
        run += __shfl(incl, kWave - 1, kWave);
    }
    return -1;
}

// First flat item of sequence t (items as in ragged_locate), or -1 when it
// lies past `limit`.  Called by a whole wave.
template <class Count>
__device__ int ragged_first(int t, int limit, Count count) {
    const int lane = threadIdx.x % kWave;
    int run = 0;
    for (int s0 = 0; s0 < t && run <= limit; s0 += kWave) {
        const int s = s0 + lane;
        const int n0 = count(s < t ? s : t - 1);
        run += wave_sum_i(s < t ? n0 : 0);
    }
    return run <= limit ? __builtin_amdgcn_readfirstlane(run) : -1;
}

}  // namespace vz

// ---- launchers (one per kernel family), called by the host API -------------
struct VzDecodeArgs {
    const void* q; const void* k_new; const void* v_new;
    void* k_cache; void* v_cache; float* score; int32_t* pos; void* out;
    int32_t len, next_pos; float gamma, sm_scale;
    int32_t L, Hq, Hkv, d, cap, dtype;
    void* ws; size_t ws_bytes;
    // ragged batch (rag.n > 0): len, next_pos and cap above are unused; q, out
    // are [n][L][Hq][d], k_new, v_new [n][L][Hkv][d], planes hold rag.total slots
    VzRagged rag;
    // a single sequence on the whole-range path in one part
    // (vz_decode_evicts): the eviction of the len + 1 slots the step leaves
    // runs in the decode kernel (ev = 1), with these arguments; ev_n is the
    // eviction workspace's move-count array
    int32_t ev, ev_budget, ev_sink, ev_M;
    int32_t* ev_kept;
    int32_t* ev_n;
};

struct VzEvictArgs {
    void* k_cache; void* v_cache; float* score; int32_t* pos;
    int32_t len, budget, n_sink, n_recent, next_pos;
    int32_t* kept_pos_out;
    int32_t L, Hkv, d, cap, dtype;
    void* ws; size_t ws_bytes;
    // ragged batch (rag.n > 0): len, budget, next_pos and cap above are unused;
    // kept_pos_out is [L][rag.total] (sequence s from slot base[s]); new_len_out
    // receives min(len, budget) per sequence
    VzRagged rag;
    int32_t* new_len_out;
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
struct VzFuseRaggedArgs {
    const void* k_in; const void* v_in;
    const int64_t* in_base; const int32_t* T_in;
    const int32_t* span_off; const int64_t* off_base; const int32_t* n_spans;
    const void* anchor_k; const void* anchor_v;
    void* k_out; void* v_out; float* score_out; int32_t* pos_out;
    const int64_t* seq_base; const int32_t* cap; int32_t* status;
    int32_t n_seqs; int64_t total_in, total_off, total; int32_t max_spans;
    int32_t L, Hkv, d, dtype;
};
hipError_t vz_launch_fuse_ragged(const VzFuseRaggedArgs& a, hipStream_t stream);
// Decode sizing: plane = slots per (layer, KV head) plane (cap, or the total
// of a ragged batch); n_seqs = 0 for a single sequence.
size_t vz_decode_ws_bytes(int32_t L, int32_t Hq, int32_t Hkv, int32_t d, int64_t plane, int32_t n_seqs);
// decode workspace: a header of vz_decode_hdr_bytes(L) bytes, then
// path-specific scratch
size_t vz_decode_hdr_bytes(int32_t L);
bool vz_decode_fused_ok(int32_t dtype, int32_t d, int32_t Hq, int32_t Hkv, int32_t L, int64_t plane, int32_t n_seqs);
size_t vz_decode_fused_ws_bytes(int32_t L, int32_t Hq, int64_t plane, int32_t n_seqs);
hipError_t vz_launch_decode_fused(const VzDecodeArgs& a, hipStream_t stream);
bool vz_decode_generic_ok(int64_t plane, int32_t n_seqs);
size_t vz_decode_generic_ws_bytes(int32_t L, int32_t Hq, int64_t plane, int32_t n_seqs);
hipError_t vz_launch_decode_generic(const VzDecodeArgs& a, hipStream_t stream);
hipError_t vz_launch_decode(const VzDecodeArgs& a, hipStream_t stream);
// Whole-range decode path (single sequence): whether a call takes it.
bool vz_decode_takes_range(const VzDecodeArgs& a);
// Workspace of the whole-range path (single sequence or ragged batch).
size_t vz_decode_range_ws_bytes(int32_t L, int32_t Hq, int32_t Hkv, int64_t plane, int32_t n_seqs);
// Whether a decode call's kernel also runs the eviction of the len + 1 slots
// it leaves (whole-range path in one part, Hkv <= 4, at most 256 moved rows).
bool vz_decode_evicts(const VzDecodeArgs& a, int32_t budget);
// A fresh nonzero tag per call (arrival counters of the whole-range path).
uint32_t vz_call_tag();
size_t vz_evict_ws_bytes(int32_t L, int64_t plane, int32_t n_seqs);
hipError_t vz_launch_evict(const VzEvictArgs& a, hipStream_t stream);
