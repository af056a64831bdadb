// Decode step (Sec. 3.1 Eq. 1-2, Sec. 3.2.2 Eq. 6), whole-range path: for a
// single-sequence call over many (layer, KV head) items, one workgroup per
// item streams every key, so no per-chunk partial results leave the chip.
// Compiled with the max-ILP machine scheduler (per-file flag of the build):
// the default one over-subscribes the 256 registers per lane and spills.
#include "decode_mfma.h"

namespace {

using namespace vz_mfma;

// ---- whole-range path: single-sequence calls over many (layer, KV head) items ----
// One workgroup of RW waves per (layer, KV head) streams every key of the
// head, so the softmax of its query heads completes inside the workgroup:
// wave w takes a contiguous run of about 1 / RW of the full 128-key chunks
// (contiguous runs stream about 7 % faster than chunks dealt round-robin to
// the waves), and wave 0 also the last, partial chunk: the first wave of each
// SIMD gets the memory pipe first and finishes tens of microseconds ahead of
// the second, so work added to it stays off the critical path.  Each wave
// keeps, per head, a running
// max, sum and output (online softmax, the output rescaled whenever the max
// grows), plus each chunk's p~ = exp2(s - m_ref) in half precision (the
// first RLDS chunks in LDS, the others in registers) and the reference max
// m_ref it was taken against.  At the end
// the waves merge their (max, sum) pairs and outputs in LDS, the workgroup
// writes its query heads' output rows, and every key's sum over those heads
// of p_hj goes to the workspace.  A fold kernel then adds the KV heads' sums
// into Eq. (6).  Compared with the chunked path there are no per-chunk
// partial outputs or probabilities in HBM and no merge launch; it needs
// enough (layer, KV head) items to occupy the GPU, one workgroup per CU.
constexpr int RW = 8;                              // waves per workgroup (256 registers per lane)
constexpr int RFULL = 8;                           // full chunks per wave
constexpr int RNCH = RFULL + 1;                    // ... plus a last chunk of at most VT keys
constexpr int RLDS = 5;                            // chunks whose p~ waits in LDS (the rest in registers)
constexpr int RANGE_MAX_KEYS = RW * RFULL * CHUNK + VT;  // 8224 keys: T = B + 1 for budgets up to 8223
constexpr int RANGE_MIN_ITEMS = 128;               // (layer, KV head) items for the whole-range path
constexpr int RO_STRIDE = D + 4;                   // padded LDS row of a wave's output (floats)

// Workspace after the header: G_sum [L][Hkv][range_row(plane)] float, the sum
// over the KV head's query heads of p_hj for every key (rows padded to whole
// chunks, so the last chunk of a row is written whole).
inline __host__ __device__ int64_t range_row(int64_t plane) { return (plane + CHUNK - 1) / CHUNK * CHUNK; }

// Row of key r (0..CHUNK-1) in a chunk's [key][head] half-precision rows
// (16 bytes each): bit 1 is flipped by bit 4, so that the 8 keys one write
// instruction covers (r = c + 4 q4 + 16 hi) start on 8 distinct 4-bank groups.
__device__ __forceinline__ int pslot(int r) { return r ^ ((r >> 3) & 2); }

template <int NW>
__global__ __launch_bounds__(64 * RW, 1) void decode_range_kernel(const FusedArgs a) {
    static_assert(RW * GMAX * RO_STRIDE * 4 <= RW * TILE_BYTES, "the merged outputs fit in the tile buffers");
    __shared__ __attribute__((aligned(16))) uint8_t s_tile[RW][TILE_BYTES];
    __shared__ float2 s_stat[RW][GMAX];
    // p~ of the first RLDS chunks of each wave, transposed: [slot(key)][head]
    // in half precision (16 bytes per key; slot() in the head-sum epilogue)
    __shared__ __attribute__((aligned(16))) uint16_t s_pt[RW][RLDS][CHUNK][GMAX];
    __shared__ __attribute__((aligned(16))) float s_mref[RW][RNCH][GMAX];  // reference max of each chunk's p~, per head (then its factor)
    __shared__ float2 s_MS[GMAX];             // the workgroup's max M and 1 / sum S, per head
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int q4 = lane >> 4, r16 = lane & 15;
    const int hi = r16 >> 3, hh = r16 & 7;
    const int Hq = a.Hq, G = Hq / NW;
    const int g = blockIdx.x, l = blockIdx.y;
    const int len = a.len, T = len + 1;
    const int n_full = T / CHUNK;            // full chunks; chunk n_full holds the other T % CHUNK keys
    const bool part = T % CHUNK != 0;
    const int c0 = __builtin_amdgcn_readfirstlane(w * n_full / RW);  // the wave's full chunks: [c0, c0 + my_full)
    const int my_full = __builtin_amdgcn_readfirstlane((w + 1) * n_full / RW - c0);
    const int my_chunks = my_full + (w == 0 && part ? 1 : 0);
    // Chunk of the wave's slot k.  Wave 0 has the fewest full chunks
    // (n_full / RW), so the partial chunk is at most its slot RFULL, and there
    // only when n_full = RW * RFULL, where the host limit leaves it <= VT keys.
    auto chunk_of = [&](int k) { return k < my_full ? c0 + k : n_full; };
    const size_t head_base = (static_cast<size_t>(l) * NW + g) * a.plane * D;
    uint16_t* Kh = a.k_cache + head_base;
    uint16_t* Vh = a.v_cache + head_base;

    // Eq. (1) first: the wave whose chunks hold slot len (the partial chunk's
    // wave 0, else the last wave) writes the new row before any of its loads,
    // so every key is read from the cache alike.
    if (w == (part ? 0 : RW - 1)) {
        const uint16_t* kn = a.k_new + (static_cast<size_t>(l) * NW + g) * D;
        const uint16_t* vn = a.v_new + (static_cast<size_t>(l) * NW + g) * D;
        if (lane < 16)
            *reinterpret_cast<uint4*>(Kh + static_cast<size_t>(len) * D + 8 * lane) =
                *reinterpret_cast<const uint4*>(kn + 8 * lane);
        else if (lane < 32)
            *reinterpret_cast<uint4*>(Vh + static_cast<size_t>(len) * D + 8 * (lane - 16)) =
                *reinterpret_cast<const uint4*>(vn + 8 * (lane - 16));
        if (g == 0 && lane == 0) a.pos[static_cast<size_t>(l) * a.plane + len] = a.next_pos;
        __threadfence_block();
    }

    // Tile t of the wave (t = 8 k + j): chunk chunk_of(k), K tiles j = 0..3 and
    // V tiles j = 4..7, 32 rows each.  Two tiles are in flight, in register
    // sets t & 1.  A tile past the wave's chunks has an empty descriptor: its
    // loads return zero and touch no memory.
    const int lane_off = q4 * (D * 2) + 16 * r16;
    uint4 stg[2][8];
    auto load_tile = [&](int k, int j, uint4 (&dst)[8]) {
        const bool live = k < my_chunks;
        const int c = live ? chunk_of(k) : 0;
        const int nk = live ? min(CHUNK, T - c * CHUNK) : 0;
        const int u = j & 3;
        const int rows = nk - VT * u > 0 ? nk - VT * u : 0;
        const uint16_t* base = (j < 4 ? Kh : Vh) + (static_cast<size_t>(c) * CHUNK + VT * u) * D;
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, rows * D * 2, kBufferDword3);
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, lane_off + 4 * m * (D * 2), 0, 0);
            __builtin_memcpy(&dst[m], &v, 16);
        }
    };
    load_tile(0, 0, stg[0]);
    load_tile(0, 1, stg[1]);

    uint8_t* const buf = s_tile[w];
    uint8_t* const kw = buf + q4 * KSTRIDE + 16 * r16;
    uint8_t* const vw = buf + q4 * VSTRIDE + 16 * r16;
    const uint8_t* const kr = buf + r16 * KSTRIDE + 16 * q4;
    const uint8_t* const vr = buf + (4 * q4 + (r16 >> 2)) * VSTRIDE + 16 * ((r16 & 3) >> 1) + 8 * (r16 & 1);

    uint4 qv[KSTEPS];  // B operand: Q^T, column r16 = query head (zero past G)
    {
        const int hq = r16 < G ? r16 : 0;
        const uint16_t* qrow = a.q + (static_cast<size_t>(l) * Hq + g * G + hq) * D + 8 * q4;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
            const uint4 v = *reinterpret_cast<const uint4*>(qrow + 32 * s);
            qv[s] = (r16 < G) ? v : make_uint4(0, 0, 0, 0);
        }
    }

    // Running state of head hh (columns r16 and r16 + 8 of the outputs hold
    // the same head): max, sum of exp2 relative to it, output relative to it.
    float m_w = -INFINITY, l_w = 0.f;
    f32x4 oacc[DTILES];
#pragma unroll
    for (int n = 0; n < DTILES; ++n) oacc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    // p~ of chunks RLDS.. RFULL - 1 in registers (half pairs); a wave's
    // chunk RFULL exists only as the last chunk of a cache with more than
    // RW * RFULL full chunks, which has at most VT keys: one 32-key tile.
    uint32_t pst[RFULL - RLDS][2 * PAIRS];
    uint32_t pst_last[2];

#pragma unroll
    for (int k = 0; k < RNCH; ++k) {
        if (k < my_chunks) {
        const int c = chunk_of(k);
        const int nk = min(CHUNK, T - c * CHUNK);
        // ---- pass 1: logits S^T = K Q^T ----
        float sp[PAIRS][4];
#pragma unroll
        for (int u = 0; u < PAIRS; ++u) {
#pragma unroll
            for (int m = 0; m < 8; ++m) *reinterpret_cast<uint4*>(kw + 4 * KSTRIDE * m) = stg[u & 1][m];
            load_tile(k, u + 2, stg[u & 1]);  // K2, K3, then V0, V1
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the tile is in LDS
            f32x4 acc[2];
#pragma unroll
            for (int ti = 0; ti < 2; ++ti) {
                acc[ti] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < KSTEPS; ++s) {
                    const uint4 av = *reinterpret_cast<const uint4*>(kr + 16 * KSTRIDE * ti + 64 * s);
                    acc[ti] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av), as_bf16x8(qv[s]), acc[ti], 0, 0, 0);
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float odd = ror8(acc[1][i]);
                const float v = hi ? odd : acc[0][i];
                const int key = VT * u + 16 * hi + 4 * q4 + i;
                sp[u][i] = (key < nk) ? v * a.scale_log2 : -INFINITY;
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the next tile is stored
        }
        // ---- online softmax: the new running max, p~ against it ----
        float m_c = -INFINITY;
#pragma unroll
        for (int u = 0; u < PAIRS; ++u)
#pragma unroll
            for (int i = 0; i < 4; ++i) m_c = fmaxf(m_c, sp[u][i]);
        m_c = fmaxf(m_c, __shfl_xor(m_c, 16, 64));
        m_c = fmaxf(m_c, __shfl_xor(m_c, 32, 64));
        m_c = fmaxf(m_c, ror8(m_c));
        const float m_new = fmaxf(m_w, m_c);
        const float alpha = m_w == -INFINITY ? 0.f : exp2f(m_w - m_new);
        float l_c = 0.f;
#pragma unroll
        for (int u = 0; u < PAIRS; ++u)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                sp[u][i] = exp2f(sp[u][i] - m_new);
                l_c += sp[u][i];
            }
        l_c += __shfl_xor(l_c, 16, 64);
        l_c += __shfl_xor(l_c, 32, 64);
        l_c += ror8(l_c);
        l_w = fmaf(l_w, alpha, l_c);
        m_w = m_new;
        if (q4 == 0 && hi == 0) s_mref[w][k][hh] = m_new;
#pragma unroll
        for (int n = 0; n < DTILES; ++n) oacc[n] *= alpha;
        // ---- pass 2: O^T += V^T P^T ----
#pragma unroll
        for (int u = 0; u < PAIRS; ++u) {
#pragma unroll
            for (int m = 0; m < 8; ++m) *reinterpret_cast<uint4*>(vw + 4 * VSTRIDE * m) = stg[u & 1][m];
            if (u < 2) load_tile(k, u + 6, stg[u & 1]);  // V2, V3
            else load_tile(k + 1, u - 2, stg[u & 1]);    // the next chunk's K0, K1
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
                s16x4 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(vr + 32 * n));
                s16x4 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4*)(vr + 16 * VSTRIDE + 32 * n));
                uint4 bw;
                __builtin_memcpy(&bw.x, &b0, 8);
                __builtin_memcpy(&bw.z, &b1, 8);
                oacc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(bw), pa, oacc[n], 0, 0, 0);
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the next tile is stored
        }
        uint32_t pk[2 * PAIRS];
#pragma unroll
        for (int u = 0; u < PAIRS; ++u) {
            pk[2 * u] = pack_f16x2(sp[u][0], sp[u][1]);
            pk[2 * u + 1] = pack_f16x2(sp[u][2], sp[u][3]);
        }
        if (k < RLDS) {
            // written as [key][head] rows now, while the wave waits for memory
            // anyway, so that the epilogue only reads whole rows
            uint16_t* const pt = &s_pt[w][k][0][0];
#pragma unroll
            for (int u = 0; u < PAIRS; ++u)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    pt[pslot(VT * u + 16 * hi + 4 * q4 + i) * GMAX + hh] =
                        static_cast<uint16_t>(pk[2 * u + (i >> 1)] >> (16 * (i & 1)));
        } else if (k < RFULL) {
#pragma unroll
            for (int i = 0; i < 2 * PAIRS; ++i) pst[k - RLDS][i] = pk[i];
        } else {
            pst_last[0] = pk[0];
            pst_last[1] = pk[1];
        }
        }
    }

    // ---- the workgroup's statistics per head: max M and 1 / sum ----
    if (q4 == 0 && hi == 0) s_stat[w][hh] = make_float2(m_w, l_w);
    __syncthreads();
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < RW; ++v) M = fmaxf(M, s_stat[v][hh].x);
    float S = 0.f;
#pragma unroll
    for (int v = 0; v < RW; ++v) {
        const float2 st = s_stat[v][hh];
        S = fmaf(st.y, st.x == -INFINITY ? 0.f : exp2f(st.x - M), S);
    }
    const float inv_S = 1.0f / S;
    if (w == 0 && q4 == 0 && hi == 0) s_MS[hh] = make_float2(M, inv_S);  // read after the next barrier

    // ---- output rows: the waves' outputs, rescaled, summed in wave order ----
    float* const s_o = reinterpret_cast<float*>(&s_tile[0][0]);  // [RW][GMAX][RO_STRIDE]
    {
        const float fo = m_w == -INFINITY ? 0.f : exp2f(m_w - M) * inv_S;
        if (r16 < G) {
#pragma unroll
            for (int n = 0; n < DTILES; ++n)
                *reinterpret_cast<f32x4*>(s_o + (w * GMAX + r16) * RO_STRIDE + 16 * n + 4 * q4) = oacc[n] * fo;
        }
    }
    __syncthreads();
    for (int e = tid; e < G * D; e += 64 * RW) {
        const int h = e / D, ch = e - h * D;
        float o = 0.f;
#pragma unroll
        for (int v = 0; v < RW; ++v) o += s_o[(v * GMAX + h) * RO_STRIDE + ch];
        a.out[(static_cast<size_t>(l) * Hq + g * G + h) * D + ch] = vz::f32_to_bf16(o);
    }

    // ---- each key's sum over this KV head's query heads of p_hj ----
    // Every chunk's p~ ends up as [slot(key)][head] half-precision rows: the
    // LDS-resident chunks were written so in the loop, the register-held ones
    // are written to the wave's (now free) tile buffer here.  Each lane then
    // reads two keys' rows and forms sum_h p~_h * f_h with f_h =
    // exp2(m_ref,h - M_h) / S_h from a per-chunk factor table.  (LDS
    // operations of a wave complete in order: no barrier between a wave's own
    // writes and reads.)
    __syncthreads();  // the output merge has read the tile buffers; s_MS is written
    float* const gsum = reinterpret_cast<float*>(a.ws + a.hdr_bytes) + (static_cast<size_t>(l) * NW + g) * range_row(a.plane);
    // factor table, in place of the reference maxima: f[k][h]
    for (int e = lane; e < RNCH * GMAX; e += 64) {
        const int k = e / GMAX, h = e - k * GMAX;
        if (k < my_chunks) {
            const float2 ms = s_MS[h];
            s_mref[w][k][h] = h < G ? exp2f(s_mref[w][k][h] - ms.x) * ms.y : 0.f;
        }
    }
    uint16_t* const scratch = reinterpret_cast<uint16_t*>(s_tile[w]);  // [CHUNK][GMAX] halves
#pragma unroll 1
    for (int k = 0; k < my_chunks; ++k) {
        const uint16_t* rows = &s_pt[w][k < RLDS ? k : 0][0][0];
        if (k >= RLDS) {
            uint32_t pk[2 * PAIRS];
            pk[0] = pst_last[0];
            pk[1] = pst_last[1];
#pragma unroll
            for (int i = 2; i < 2 * PAIRS; ++i) pk[i] = 0;  // keys past the cache: p~ = 0
#pragma unroll
            for (int r = 0; r < RFULL - RLDS; ++r)  // register slots: fixed indexes, wave-uniform choice
                if (k == RLDS + r) {
#pragma unroll
                    for (int i = 0; i < 2 * PAIRS; ++i) pk[i] = pst[r][i];
                }
#pragma unroll
            for (int u = 0; u < PAIRS; ++u)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    scratch[pslot(VT * u + 16 * hi + 4 * q4 + i) * GMAX + hh] =
                        static_cast<uint16_t>(pk[2 * u + (i >> 1)] >> (16 * (i & 1)));
            rows = scratch;
        }
        const float4 fa = *reinterpret_cast<const float4*>(&s_mref[w][k][0]);
        const float4 fb = *reinterpret_cast<const float4*>(&s_mref[w][k][4]);
        const float fk[GMAX] = {fa.x, fa.y, fa.z, fa.w, fb.x, fb.y, fb.z, fb.w};
        float y[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const uint4 r = *reinterpret_cast<const uint4*>(rows + pslot(2 * lane + e) * GMAX);
            const uint32_t wd[4] = {r.x, r.y, r.z, r.w};
            float acc = 0.f;
#pragma unroll
            for (int h = 0; h < GMAX; ++h)
                acc = fmaf(f16_to_f32(static_cast<uint16_t>(wd[h >> 1] >> (16 * (h & 1)))), fk[h], acc);
            y[e] = acc;
        }
        *reinterpret_cast<float2*>(gsum + chunk_of(k) * CHUNK + 2 * lane) = make_float2(y[0], y[1]);
    }
}

// Fold kernel of the whole-range path, thread = key: Eq. (6) with the KV
// heads' sums added in head order (the new slot starts from 0).
constexpr int RFOLD_THREADS = 256;
template <int NW>
__global__ __launch_bounds__(RFOLD_THREADS) void decode_range_fold_kernel(const FusedArgs a) {
    const int l = blockIdx.y;
    const int len = a.len;
    const int j = min(static_cast<int>(blockIdx.x) * RFOLD_THREADS + static_cast<int>(threadIdx.x), len);
    const int64_t row = range_row(a.plane);
    const float* gs = reinterpret_cast<const float*>(a.ws + a.hdr_bytes) + static_cast<size_t>(l) * NW * row + j;
    float* const sc = a.score + static_cast<size_t>(l) * a.plane + j;
    const float a_ld = *sc;
    float acc = gs[0];
#pragma unroll
    for (int g = 1; g < NW; ++g) acc += gs[g * row];
    const float a_old = j < len ? a_ld : 0.f;  // zero pad of Eq. (6) for the new slot
    if (static_cast<int>(blockIdx.x) * RFOLD_THREADS + static_cast<int>(threadIdx.x) <= len) *sc = fmaf(a.gamma, a_old, acc);
}

template <int NW>
hipError_t launch_range(const FusedArgs& a, bool fold, hipStream_t stream) {
    hipLaunchKernelGGL((decode_range_kernel<NW>), dim3(NW, a.L), dim3(64 * RW), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !fold) return e;
    hipLaunchKernelGGL((decode_range_fold_kernel<NW>), dim3((a.len + RFOLD_THREADS) / RFOLD_THREADS, a.L),
                       dim3(RFOLD_THREADS), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

bool vz_decode_range_ok(int32_t len, int32_t L, int32_t Hkv) {
    return static_cast<int64_t>(len) + 1 <= RANGE_MAX_KEYS && static_cast<int64_t>(L) * Hkv >= RANGE_MIN_ITEMS;
}

hipError_t vz_launch_decode_range(const FusedArgs& a, int32_t Hkv, bool fold, hipStream_t stream) {
    switch (Hkv) {
        case 1: return launch_range<1>(a, fold, stream);
        case 2: return launch_range<2>(a, fold, stream);
        case 4: return launch_range<4>(a, fold, stream);
        case 8: return launch_range<8>(a, fold, stream);
        default: return hipErrorInvalidValue;
    }
}

int64_t vz_range_sum_row(int64_t plane) { return range_row(plane); }
