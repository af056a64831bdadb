// Definitions shared by the MFMA decode kernels (bfloat16 caches, d = 128,
// at most 8 query heads per KV head): tile geometry, operand helpers and the
// kernel arguments.  Included by the chunked path (decode_fused.hip) and the
// whole-range path (decode_range.hip).
#pragma once

#include <math.h>

#include "vz_internal.h"

namespace vz_mfma {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr int D = 128;
constexpr int GMAX = 8;                // query heads per KV head served here
constexpr int TILES = 8;               // 16-key MFMA tiles per chunk
constexpr int PAIRS = TILES / 2;       // packed tile pairs = 32-key tiles
constexpr int CHUNK = 16 * TILES;      // keys per chunk (at most)
constexpr int VT = 32;                 // keys per staged tile
constexpr int KSTEPS = D / 32;         // MFMA k-steps over the channels
constexpr int DTILES = D / 16;         // output column tiles
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kRor8 = 0x128;           // DPP row_ror:8 (swap the halves of each 16-lane row)
constexpr int kBufferDword3 = 0x00020000;  // raw buffer descriptor word 3 (32-bit data format)

// Staged tiles are 32 rows of 256 bytes with padded row strides, so that every
// LDS address is one per-lane base plus an immediate (bank analysis in the
// design notes): K rows 272 bytes apart (16 rows at one 16-byte column fall on
// 16 distinct bank groups), V rows 288 bytes apart (4 rows x 32 bytes of a
// transposed read fall on distinct banks).  (The chunked attend kernel loads
// its K tiles straight into the MFMA operand layout instead; only its V
// tiles go through LDS.)
constexpr int KSTRIDE = 256 + 16;
constexpr int VSTRIDE = 256 + 32;
constexpr int TILE_BYTES = VT * VSTRIDE;

// Chunk c of a sequence of T keys: keys [c * CHUNK, min((c + 1) * CHUNK, T)),
// so every chunk is full except the last (the remainder of T / CHUNK).
__device__ __forceinline__ int chunk_begin(int c) { return c * CHUNK; }
__device__ __forceinline__ int chunk_keys(int c, int T) { return min(CHUNK, T - c * CHUNK); }

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) {
    bf16x8_t r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

__device__ __forceinline__ float ror8(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kRor8, 0xF, 0xF, false));
}

// Two floats to packed bfloat16 (low half a), round to nearest even: one
// v_cvt_pk_bf16_f32 on gfx950 (the same bits as vz::f32_to_bf16 for finite
// values).  Used for the P operand of the P.V products and for the stored
// probabilities p~, which keep 8 significant bits at any magnitude (no
// subnormal range to fall into, unlike half precision).
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    const bf16x2_t r = __builtin_convertvector(f32x2_t{a, b}, bf16x2_t);
    uint32_t u;
    __builtin_memcpy(&u, &r, 4);
    return u;
}
// The low and high bfloat16 of a packed pair, widened.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Kernel arguments shared by the decode launches.  A single-sequence call
// has rag.n == 0 and takes len, next_pos and n_chunks from here; a ragged
// call reads them per sequence, and n_chunks is then its grid extent per
// layer (nc_max).
struct FusedArgs {
    const uint16_t* q;
    const uint16_t* k_new;
    const uint16_t* v_new;
    uint16_t* k_cache;
    uint16_t* v_cache;
    int32_t* pos;
    float* score;
    uint16_t* out;
    uint8_t* ws;
    int32_t len, next_pos;  // single sequence
    int32_t n_chunks;       // single sequence
    int32_t nc_max;         // chunk rows of the partials per layer (grid bound for a ragged call)
    int32_t Hq, L, hdr_bytes;
    int64_t plane;          // slots per (layer, KV head) plane
    float scale_log2, gamma;
    VzRagged rag;
    // whole-range path: a single sequence's parts (n_parts = 1: one part of
    // every key; else parts of part_keys keys, the last one shorter), and the
    // bounds of a ragged call's work tables (R parts, FB fold blocks)
    int32_t n_parts, part_keys, R, FB;
    int32_t MB;   // a ragged call's bound on sequences in several parts
    int32_t cus;  // compute units of the device (the choice of parts)
    // whole-range path, a single sequence in one part: the last workgroup of
    // each layer to finish (elected on the arrival counters cnt[L] with the
    // call's tag) folds the scores (Eq. 6) and, when ev != 0, runs the
    // eviction of the len + 1 slots (Sec. 3.2.2 Eq. 7-9) with budget ev_budget,
    // ev_sink sinks, an ev_M recent window, optional kept positions ev_kept
    // [L][ev_budget] and the move counts ev_n [L] of the eviction workspace
    uint64_t* cnt;
    uint32_t tag;
    int32_t ev, ev_budget, ev_sink, ev_M;
    int32_t* ev_kept;
    int32_t* ev_n;
};

}  // namespace vz_mfma

// Whole-range path (decode_range.hip): whether a call over L layers, Hkv KV
// heads and n_seqs sequences (0: a single sequence) takes it, and its
// launches (a single sequence: a.len, a.next_pos; a ragged batch: a.rag).
bool vz_decode_range_ok(int32_t L, int32_t Hkv, int32_t n_seqs);
hipError_t vz_launch_decode_range(const vz_mfma::FusedArgs& a, int32_t Hkv, hipStream_t stream);
// Whether a single sequence of len resident keys is one part (one launch of
// the range kernel, which also folds the scores, and evicts when asked).
bool vz_decode_range_whole(int32_t len);
