// Decode step (Sec. 3.1 Eq. 1-2, Sec. 3.2.2 Eq. 6) for bfloat16 caches with
// d = 128 and at most 8 query heads per KV head.  Two launches cover every
// layer: the attend kernel (attention on the matrix cores and the
// decayed-score fold from registers) and a small combine kernel (the output
// rows from the per-chunk partials).
//
// Attend kernel: work item = (layer, key chunk of <= 256 keys).  A workgroup
// has one wave per KV head; wave g streams K and V rows of head g over the
// chunk:
//   pass 1  S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (M = 16 keys, N = 16
//           query-head columns of which n_q/n_kv <= 8 are used, K = 32
//           channels).  K tiles of 32 rows are loaded fully coalesced (4 whole
//           rows per 1 KB instruction), stored to LDS with an XOR swizzle on
//           the row index, and read back with ds_read_b128 in the A-operand
//           layout, bank-conflict free.  One tile is in flight while the
//           previous one is multiplied.  The logits of an odd 16-key tile are
//           moved into the unused head columns 8..15 of the even tile's
//           registers (DPP row rotate by 8), so 256 keys x 8 heads take 32
//           registers per lane.
//   stats   chunk-local max and sum per head; the registers then hold
//           p~ = exp(s - m_chunk).  Each (max, sum) pair is published to the
//           workspace at once with one 64-bit store; a sum is at least 1 for
//           a non-empty chunk, so a zero sum marks a pair not yet published.
//   pass 2  O += P V: V tiles of 32 keys take the same coalesced path into
//           LDS (another swizzle) and are read back with ds_read_b64_tr_b16
//           directly in the B-operand layout; P is rebuilt from the packed p~
//           registers with one row rotate.  The partial O goes to the
//           workspace for the combine kernel.
//   fold    by now the other chunks of the layer have normally published
//           their statistics too (the wait is for their pass 1 only); each
//           wave polls the pairs of its own heads until none is zero, merges
//           them into the layer's (max, sum) per head and folds
//               A[j] = gamma * A[j] + sum_h exp(s_hj - m_h) / l_h
//           for its own keys from the p~ still in registers -- no logit ever
//           goes to HBM.
// Work items are taken in ticket order (one atomic per workgroup), so the
// chunks of a layer start together whatever order the hardware dispatches
// workgroups in.  A chunk waits only for chunks of its layer that already
// hold a ticket and never wait themselves before publishing, and the number
// of chunks per layer is kept below the number of workgroups that can be
// resident, so every wait ends; it is also bounded in time (on expiry the
// kernel flags an error in the workspace and finishes).  Statistics move
// through device-scope atomic stores and loads, coherent across the per-XCD
// L2 caches, so no cache-wide flush is needed.  The combine kernel, which
// runs after every attend workgroup has finished, zeroes the pairs it has
// read and the ticket, so the workspace is ready for the next call.
#include <math.h>

#include "vz_internal.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr int D = 128;
constexpr int GMAX = 8;                // query heads per KV head served here
constexpr int TILES = 16;              // 16-key MFMA tiles per chunk
constexpr int PAIRS = TILES / 2;       // packed tile pairs = 32-key tiles
constexpr int CHUNK = 16 * TILES;      // keys per chunk (at most)
constexpr int VT = 32;                 // keys per staged tile
constexpr int KSTEPS = D / 32;         // MFMA k-steps over the channels
constexpr int DTILES = D / 16;         // output column tiles
constexpr float kLog2e = 1.4426950408889634f;
constexpr uint64_t kWaitTicks = 20000000ull;  // 0.2 s of the 100 MHz constant clock
constexpr int kRor8 = 0x128;           // DPP row_ror:8 (swap the halves of each 16-lane row)
constexpr int kBufferDword3 = 0x00020000;  // raw buffer descriptor word 3 (32-bit data format)

struct WsHeader {
    uint32_t ticket;
    uint32_t error;
    uint32_t pad[62];
};

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) {
    bf16x8_t r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

__device__ __forceinline__ float ror8(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kRor8, 0xF, 0xF, false));
}

// Device-scope (all XCDs) coherent 64-bit store / load of a float pair.
__device__ __forceinline__ void st_dev2(float2* p, float a, float b) {
    const uint64_t v = static_cast<uint64_t>(__float_as_uint(a)) | (static_cast<uint64_t>(__float_as_uint(b)) << 32);
    __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_dev2(const float2* p) {
    const uint64_t v =
        __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return make_float2(__uint_as_float(static_cast<uint32_t>(v)), __uint_as_float(static_cast<uint32_t>(v >> 32)));
}

// Merge two (max, sum-of-exp2) softmax partials.
__device__ __forceinline__ void merge_ml(float& m, float& l, float m2, float l2) {
    if (m2 == -INFINITY) return;
    if (m == -INFINITY) {
        m = m2;
        l = l2;
        return;
    }
    const float mn = fmaxf(m, m2);
    l = l * exp2f(m - mn) + l2 * exp2f(m2 - mn);
    m = mn;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return static_cast<uint32_t>(vz::f32_to_bf16(a)) | (static_cast<uint32_t>(vz::f32_to_bf16(b)) << 16);
}

// XOR swizzles of the 16-byte chunks of a staged row in LDS (bank analysis in
// the design notes).  K: row r of the tile.  V: row a of 4-row block b.
__device__ __forceinline__ int kswz(int r) { return r & 15; }
__device__ __forceinline__ int vswz(int a, int b) { return ((a << 1) + ((b & 1) << 3)) & 15; }

template <int NW>
__global__ __launch_bounds__(64 * NW, 2) void decode_attend_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache, float* __restrict__ score,
    int32_t* __restrict__ pos, int32_t len, int32_t next_pos, float gamma, float scale_log2, int32_t Hq,
    int32_t cap, int32_t n_chunks, int32_t nc_max, int32_t n_items, int32_t L, uint8_t* __restrict__ ws,
    int32_t hdr_bytes) {
    __shared__ uint32_t s_item;
    __shared__ __attribute__((aligned(16))) uint8_t s_tile[NW][VT * D * 2];
    __shared__ float s_psum[NW][CHUNK];

    const int tid = threadIdx.x;
    // wave-uniform values go through readfirstlane so that addresses built
    // from them stay scalar (buffer descriptors in SGPRs)
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int q4 = lane >> 4, r16 = lane & 15;
    const int hi = r16 >> 3;          // 0: even tile of a pair, 1: odd tile (packed lanes)
    const int hh = r16 & 7;           // query head of the group this lane's logits belong to
    const int G = Hq / NW;
    const int g = w;                  // KV head of this wave

    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws);
    float2* part_ml = reinterpret_cast<float2*>(ws + hdr_bytes);
    float* part_o = reinterpret_cast<float*>(ws + hdr_bytes) + 2 * L * nc_max * Hq;

    if (tid == 0) s_item = atomicAdd(&hdr->ticket, 1u);
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(static_cast<int>(s_item));
    if (item >= n_items) {  // the workspace was not zero-filled: flag it, touch nothing else
        if (tid == 0) __hip_atomic_store(&hdr->error, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int l = item / n_chunks, c = item % n_chunks;
    const int T = len + 1;
    const int k_begin = static_cast<int>(static_cast<int64_t>(c) * T / n_chunks);
    const int k_end = static_cast<int>(static_cast<int64_t>(c + 1) * T / n_chunks);
    const int nk = k_end - k_begin;
    const size_t head_base = (static_cast<size_t>(l) * NW + g) * static_cast<size_t>(cap) * D;
    uint16_t* Kh = k_cache + head_base;
    uint16_t* Vh = v_cache + head_base;

    // Eq. (1) first: the chunk holding slot len writes the new row into the
    // cache, so every key below is read from the cache the same way.
    if (len >= k_begin && len < k_end) {
        const uint16_t* kn = k_new + (l * NW + g) * D;
        const uint16_t* vn = v_new + (l * NW + g) * D;
        if (lane < 16)
            *reinterpret_cast<uint4*>(Kh + len * D + 8 * lane) = *reinterpret_cast<const uint4*>(kn + 8 * lane);
        else if (lane < 32)
            *reinterpret_cast<uint4*>(Vh + len * D + 8 * (lane - 16)) =
                *reinterpret_cast<const uint4*>(vn + 8 * (lane - 16));
        if (tid == 0) pos[l * cap + len] = next_pos;
        __threadfence_block();
    }
    __syncthreads();

    // ---------------- pass 1: logits S^T = K Q^T ----------------
    uint4 qv[KSTEPS];  // B operand: Q^T, column r16 = query head (zero past G)
    {
        const int hq = r16 < G ? r16 : 0;
        const uint16_t* qrow = q + (l * Hq + g * G + hq) * D + 8 * q4;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
            const uint4 v = *reinterpret_cast<const uint4*>(qrow + 32 * s);
            qv[s] = (r16 < G) ? v : make_uint4(0, 0, 0, 0);
        }
    }
    uint8_t* buf = s_tile[w];
    // Staging: instruction m of a 32-key tile reads rows 4m..4m+3 whole
    // (lane = row 4m + q4, 16-byte chunk r16) with buffer loads addressed by
    // 32-bit offsets from a descriptor bounded to the head's cap rows (reads
    // outside it return zero).  Rows past the chunk end are clamped to its
    // last row and masked out afterwards.
    const int region = cap * D * 2;
    const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(Kh, 0, region, kBufferDword3);
    const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(Vh, 0, region, kBufferDword3);
    uint4 stg[8];
    auto load_tile = [&](const __amdgpu_buffer_rsrc_t& rs, int u) {
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            int j = k_begin + VT * u + 4 * m + q4;
            j = j < k_end ? j : k_end - 1;
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, j * (D * 2) + 16 * r16, 0, 0);
            __builtin_memcpy(&stg[m], &v, 16);
        }
    };
    // sp[u][i]: lanes with hi = 0 hold key 32u + 4 q4 + i, head hh; lanes with
    // hi = 1 hold key 32u + 16 + 4 q4 + i, head hh.
    float sp[PAIRS][4];
    load_tile(krs, 0);
#pragma unroll
    for (int u = 0; u < PAIRS; ++u) {
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const int row = 4 * m + q4;
            *reinterpret_cast<uint4*>(buf + 256 * row + 16 * (r16 ^ kswz(row))) = stg[m];
        }
        if (u + 1 < PAIRS) load_tile(krs, u + 1);
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the tile is in LDS
        f32x4 acc[2];
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) {
            const int row = 16 * ti + r16;
            acc[ti] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < KSTEPS; ++s) {
                const uint4 a = *reinterpret_cast<const uint4*>(buf + 256 * row + 16 * ((4 * s + q4) ^ kswz(row)));
                acc[ti] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(qv[s]), acc[ti], 0, 0, 0);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float odd = ror8(acc[1][i]);  // lane hi=1 receives the odd tile of head hh
            const float v = hi ? odd : acc[0][i];
            const int key = VT * u + 16 * hi + 4 * q4 + i;
            sp[u][i] = (key < nk) ? v * scale_log2 : -INFINITY;
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the next tile is stored
    }

    // ---------------- chunk statistics, published at once ----------------
    // per head hh (8 lanes share it: q4 x hi); afterwards sp holds p~ = exp2(s - m_c)
    float m_c = -INFINITY;
#pragma unroll
    for (int u = 0; u < PAIRS; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i) m_c = fmaxf(m_c, sp[u][i]);
    m_c = fmaxf(m_c, __shfl_xor(m_c, 16, 64));
    m_c = fmaxf(m_c, __shfl_xor(m_c, 32, 64));
    m_c = fmaxf(m_c, ror8(m_c));
    float l_c = 0.f;
#pragma unroll
    for (int u = 0; u < PAIRS; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            sp[u][i] = exp2f(sp[u][i] - m_c);
            l_c += sp[u][i];
        }
    l_c += __shfl_xor(l_c, 16, 64);
    l_c += __shfl_xor(l_c, 32, 64);
    l_c += ror8(l_c);
    const int pbase = (l * nc_max + c) * Hq + g * G;  // < 2^31 (checked on the host)
    if (q4 == 0 && r16 < G) st_dev2(&part_ml[pbase + r16], m_c, l_c);
    load_tile(vrs, 0);

    // ---------------- pass 2: O = P V on the matrix cores ----------------
    f32x4 oacc[DTILES];
#pragma unroll
    for (int n = 0; n < DTILES; ++n) oacc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < PAIRS; ++u) {
#pragma unroll
        for (int m = 0; m < 8; ++m)
            *reinterpret_cast<uint4*>(buf + 1024 * m + 256 * q4 + 16 * (r16 ^ vswz(q4, m))) = stg[m];
        if (u + 1 < PAIRS) load_tile(vrs, u + 1);
        // A operand P: row = head r16 (rows >= G feed output rows that are never
        // stored), k-slots 8 q4 + i -> keys 32u + 4 q4 + i (i < 4) and
        // 32u + 16 + 4 q4 + i - 4 (i >= 4): the even tile is in place, the odd
        // tile comes back from the upper half of the row.
        float ev[4], od[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float x = sp[u][i];
            const float y = ror8(x);
            ev[i] = hi ? y : x;
            od[i] = hi ? x : y;
        }
        const uint4 pw = make_uint4(pack_bf16x2(ev[0], ev[1]), pack_bf16x2(ev[2], ev[3]), pack_bf16x2(od[0], od[1]),
                                    pack_bf16x2(od[2], od[3]));
        const bf16x8_t pa = as_bf16x8(pw);
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the tile is in LDS
#pragma unroll
        for (int n = 0; n < DTILES; ++n) {
            const int a = r16 >> 2;
            const int cl = 2 * n + ((r16 & 3) >> 1);
            const int half = (r16 & 1) * 8;
            const uint8_t* pa0 = buf + 1024 * q4 + 256 * a + 16 * (cl ^ vswz(a, q4)) + half;
            const uint8_t* pa1 = buf + 1024 * (4 + q4) + 256 * a + 16 * (cl ^ vswz(a, 4 + q4)) + half;
            s16x4 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(pa0));
            s16x4 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(pa1));
            uint4 bw;
            __builtin_memcpy(&bw.x, &b0, 8);
            __builtin_memcpy(&bw.z, &b1, 8);
            oacc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, as_bf16x8(bw), oacc[n], 0, 0, 0);
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the next tile is stored
    }
    // partial O (read by the combine kernel after this launch): plain stores
    {
        float* po = part_o + pbase * D;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int h = 4 * q4 + i;  // output row = query head of the group
            if (h < G) {
#pragma unroll
                for (int n = 0; n < DTILES; ++n) po[h * D + 16 * n + r16] = oacc[n][i];
            }
        }
    }

    // ---------------- fold: A[j] = gamma A[j] + sum_h p_hj ----------------
    // The chunk's old scores are loaded first, so their latency overlaps the
    // wait for the statistics.
    constexpr int KPT = (CHUNK + 64 * NW - 1) / (64 * NW);  // keys per thread
    float* lsc = score + l * cap;
    float a_old[KPT];
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
        const int k = tid + 64 * NW * i;
        const int j = k_begin + k;
        a_old[i] = (k < nk && j < len) ? lsc[j] : 0.f;
    }
    // Global (max, sum) of this wave's heads: lane (q4, hi, hh) polls head hh
    // over chunks q4 + 4 hi + 8 k, 64 chunks per round, until no pair of the
    // round is unpublished; the eight lanes of a head then merge.
    float m_h = -INFINITY, l_h = 0.f;
    {
        const float2* hrow = part_ml + l * nc_max * Hq + g * G + (hh < G ? hh : 0);
        const uint64_t t0 = wall_clock64();
        for (int base = 0; base < n_chunks; base += 64) {
            float2 v[8];
            for (;;) {
                bool ready = true;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int cc = base + q4 + 4 * hi + 8 * k;
                    v[k] = cc < n_chunks ? ld_dev2(hrow + cc * Hq) : make_float2(-INFINITY, 1.f);
                    ready = ready && v[k].y != 0.f;
                }
                if (__all(ready)) break;
                if (wall_clock64() - t0 > kWaitTicks) {
                    if (lane == 0) __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
#pragma unroll
            for (int k = 0; k < 8; ++k) merge_ml(m_h, l_h, v[k].x, v[k].y);
        }
        merge_ml(m_h, l_h, __shfl_xor(m_h, 16, 64), __shfl_xor(l_h, 16, 64));
        merge_ml(m_h, l_h, __shfl_xor(m_h, 32, 64), __shfl_xor(l_h, 32, 64));
        merge_ml(m_h, l_h, ror8(m_h), ror8(l_h));
    }
    const float fac = (hh < G) ? exp2f(m_c - m_h) / l_h : 0.f;  // p = p~ * fac
#pragma unroll
    for (int u = 0; u < PAIRS; ++u) {
        if (VT * u < nk) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float pv = sp[u][i] * fac;
                pv += __shfl_xor(pv, 1, 64);
                pv += __shfl_xor(pv, 2, 64);
                pv += __shfl_xor(pv, 4, 64);
                if (hh == 0) s_psum[w][VT * u + 16 * hi + 4 * q4 + i] = pv;
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
        const int k = tid + 64 * NW * i;
        if (k < nk) {
            float a = 0.f;
#pragma unroll
            for (int gg = 0; gg < NW; ++gg) a += s_psum[gg][k];
            lsc[k_begin + k] = gamma * a_old[i] + a;  // a_old = 0 for the new slot (zero pad of Eq. 6)
        }
    }
}

// Combine kernel: one workgroup of D threads per (layer, head):
//   o_h = sum_c O_c,h exp2(m_c,h - m_h) / l_h over the layer's chunks.
// It then zeroes the (max, sum) pairs it has read (and workgroup (0, 0) the
// ticket): the attend kernel of the next call starts from a clean workspace.
__global__ __launch_bounds__(D) void decode_combine_kernel(uint8_t* __restrict__ ws, uint16_t* __restrict__ out,
                                                           int32_t Hq, int32_t n_chunks, int32_t nc_max, int32_t L,
                                                           int32_t hdr_bytes) {
    __shared__ float s_w[256];
    __shared__ float s_m, s_l;
    const int h = blockIdx.x, l = blockIdx.y, tid = threadIdx.x;
    float2* ml = reinterpret_cast<float2*>(ws + hdr_bytes) + l * nc_max * Hq + h;
    const float* po = reinterpret_cast<const float*>(ws + hdr_bytes) + 2 * L * nc_max * Hq + (l * nc_max * Hq + h) * D;
    if (tid < 64) {  // wave 0: global (max, sum) of the head over the chunks
        float m = -INFINITY, s = 0.f;
        for (int cc = tid; cc < n_chunks; cc += 64) {
            const float2 v = ml[cc * Hq];
            merge_ml(m, s, v.x, v.y);
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) merge_ml(m, s, __shfl_xor(m, o, 64), __shfl_xor(s, o, 64));
        if (tid == 0) {
            s_m = m;
            s_l = s;
        }
    }
    __syncthreads();
    const float m = s_m, inv_l = 1.0f / s_l;
    for (int cc = tid; cc < n_chunks; cc += D) s_w[cc] = exp2f(ml[cc * Hq].x - m) * inv_l;
    __syncthreads();
    for (int cc = tid; cc < n_chunks; cc += D) ml[cc * Hq] = make_float2(0.f, 0.f);
    if (h == 0 && l == 0 && tid == 0) reinterpret_cast<WsHeader*>(ws)->ticket = 0u;
    float acc = 0.f;
#pragma unroll 8
    for (int cc = 0; cc < n_chunks; ++cc) acc += s_w[cc] * po[cc * Hq * D + tid];
    out[(l * Hq + h) * D + tid] = vz::f32_to_bf16(acc);
}

}  // namespace

// ---- sizing shared with the host API ----
size_t vz_decode_hdr_bytes(int32_t L) {
    (void)L;
    return sizeof(WsHeader);
}

int32_t vz_decode_fused_chunks(int32_t T) { return (T + CHUNK - 1) / CHUNK; }

bool vz_decode_fused_ok(int32_t dtype, int32_t d, int32_t Hq, int32_t Hkv, int32_t cap, int32_t L) {
    if (dtype != VZ_BF16 || d != D) return false;
    if (!(Hkv == 1 || Hkv == 2 || Hkv == 4 || Hkv == 8)) return false;
    if (Hq % Hkv != 0 || Hq / Hkv > GMAX) return false;
    // 32-bit element offsets inside the kernels: partials, scores, positions,
    // outputs, one head's rows
    const int64_t ncm = vz_decode_fused_chunks(cap);
    if (static_cast<int64_t>(L) * ncm * Hq * (D + 2) >= (int64_t(1) << 31)) return false;
    if (static_cast<int64_t>(L) * cap >= (int64_t(1) << 31)) return false;
    if (static_cast<int64_t>(cap) * D * 2 >= (int64_t(1) << 31)) return false;
    if (static_cast<int64_t>(L) * Hq * D >= (int64_t(1) << 31)) return false;
    return ncm <= 256;  // chunks of one layer must fit on the GPU at once
}

size_t vz_decode_fused_ws_bytes(int32_t L, int32_t Hq, int32_t cap) {
    const size_t ncm = static_cast<size_t>(vz_decode_fused_chunks(cap));
    return vz_decode_hdr_bytes(L) + static_cast<size_t>(L) * ncm * Hq * (sizeof(float2) + sizeof(float) * D);
}

hipError_t vz_launch_decode_fused(const VzDecodeArgs& a, hipStream_t stream) {
    const int T = a.len + 1;
    const int n_chunks = vz_decode_fused_chunks(T);
    const int nc_max = vz_decode_fused_chunks(a.cap);
    const int n_items = a.L * n_chunks;
    const float scale = (a.sm_scale > 0.f ? a.sm_scale : 1.0f / sqrtf(static_cast<float>(D))) * kLog2e;
    const int hdr = static_cast<int>(vz_decode_hdr_bytes(a.L));
    auto* ws = static_cast<uint8_t*>(a.ws);
#define VZ_LAUNCH_ATTEND(NW)                                                                                     \
    hipLaunchKernelGGL((decode_attend_kernel<NW>), dim3(n_items), dim3(64 * NW), 0, stream,                     \
                       static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k_new),                \
                       static_cast<const uint16_t*>(a.v_new), static_cast<uint16_t*>(a.k_cache),                \
                       static_cast<uint16_t*>(a.v_cache), a.score, a.pos, a.len, a.next_pos, a.gamma, scale,    \
                       a.Hq, a.cap, n_chunks, nc_max, n_items, a.L, ws, hdr)
    switch (a.Hkv) {
        case 1: VZ_LAUNCH_ATTEND(1); break;
        case 2: VZ_LAUNCH_ATTEND(2); break;
        case 4: VZ_LAUNCH_ATTEND(4); break;
        case 8: VZ_LAUNCH_ATTEND(8); break;
        default: return hipErrorInvalidValue;
    }
#undef VZ_LAUNCH_ATTEND
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(decode_combine_kernel, dim3(a.Hq, a.L), dim3(D), 0, stream, ws,
                       static_cast<uint16_t*>(a.out), a.Hq, n_chunks, nc_max, a.L, hdr);
    return hipGetLastError();
}
