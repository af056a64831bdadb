// Decode step (Sec. 3.1 Eq. 1-2, Sec. 3.2.2 Eq. 6) for bfloat16 caches with
// d = 128 and at most 8 query heads per KV head, chunked path.  Three
// launches cover every layer: the attend kernel streams the cache once and
// leaves per-chunk partial results in the workspace; the output and fold
// kernels merge them into the output rows and the decayed scores.  No
// workgroup ever waits for another.  Single-sequence calls with enough
// (layer, KV head) items and a short enough cache go to the whole-range path
// (decode_range.hip) instead.
//
// Attend kernel: work item = (layer, key chunk of <= 128 keys, KV head), a
// workgroup of four waves, one 32-key tile each (the query rows and the K
// and V tiles of a wave are requested at once: one memory round trip per
// chunk).
//   logits  S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (M = 16 keys, N = 16
//           query-head columns of which n_q/n_kv <= 8 are used, K = 32
//           channels).  K tiles of 32 rows are loaded straight into the
//           A-operand layout (each 1 KB instruction reads 64-byte pieces of
//           16 rows) and used from registers.  The logits
//           of the odd 16-key half of a tile are moved into the unused head
//           columns 8..15 (DPP row rotate by 8), so 32 keys x 8 heads take 4
//           registers per lane.
//   stats   the chunk's max m_c per head (the four waves' maxima through
//           LDS); p~ = exp2(s - m_c) and the sum l_c of exp2 per head.
//           (m_c, l_c) and p~ (bfloat16) go to the workspace.
//   P V     V tiles take the same coalesced path into LDS and are read back
//           with ds_read_b64_tr_b16 directly in the B-operand layout; P is
//           rebuilt from p~ with one row rotate.  The four waves' O (fp32)
//           are summed in wave order through LDS; O_c (relative to m_c) goes
//           to the workspace in bfloat16.
// Output kernel: per (head, layer), the output row merged from the chunk
// partials, and the layer's (max, sum) of the head.  Fold kernel: per (chunk,
// layer), the chunk's scores A[j] = gamma A[j] + sum_h p_hj from p~ and one
// factor per head.
#include <atomic>
#include <random>
#include <type_traits>

#include "decode_mfma.h"
#include "select.h"

namespace {

using namespace vz_mfma;

// Decode workspace header: 256 reserved bytes (a ragged call keeps its table
// sizes there), then one arrival counter per layer (whole-range path, zero
// after every call), padded to 256 bytes.
constexpr size_t kHeaderBytes = 256;

// Per-chunk partial results in the workspace, after the header:
//   ml [L][nc_max][Hq]        float2     chunk max m_c and sum l_c of exp2, per head
//   o  [L][nc_max][Hq][D]     bfloat16   O_c relative to m_c
//   p  [L][nc_max][Hq][CHUNK] bfloat16   p~ = exp2(s - m_c) per key of the chunk
//   layer [S][L][Hq]          float2     the layer's max M and 1 / sum S, per head
//                                        (S = sequences of the call)
template <typename B>
struct PartialsT {
    using F2 = typename std::conditional<std::is_const<B>::value, const float2, float2>::type;
    using U16 = typename std::conditional<std::is_const<B>::value, const uint16_t, uint16_t>::type;
    F2* ml;
    U16* o;
    U16* p;
    F2* layer;
    __device__ PartialsT(B* ws, int hdr_bytes, int L, int nc_max, int Hq) {
        const size_t n = static_cast<size_t>(L) * nc_max * Hq;
        ml = reinterpret_cast<F2*>(ws + hdr_bytes);
        o = reinterpret_cast<U16*>(ml + n);
        p = o + n * D;
        layer = reinterpret_cast<F2*>(p + n * CHUNK);
    }
};
using Partials = PartialsT<uint8_t>;
using ConstPartials = PartialsT<const uint8_t>;

// Chunks of sequence s in a ragged call (0 when it cannot be served).
__device__ __forceinline__ int ragged_chunks(const VzRagged& r, int s) {
    return vz::ragged_decode_status(r, s) == VZ_OK ? (r.len[s] + CHUNK) / CHUNK : 0;
}

// The sequence a work item belongs to, resolved at the top of every kernel.
struct SeqItem {
    int s;           // sequence (0 for a single-sequence call)
    int len, next_pos;
    int n_chunks;    // chunks of the sequence
    int first;       // its first chunk row in the partials
    int64_t base;    // its first slot in the planes
};

// Flat chunk f of a ragged call, found by a whole wave: each lane loads one
// sequence's values (64 sequences per round), a wave scan of their chunk
// counts finds the owner of f, and the owner's values are forwarded from the
// lane that loaded them, so the kernel waits for one round of loads.  False
// when f lies past the call's chunks (or past the nc_max rows).
__device__ __forceinline__ bool locate_ragged_chunk(const FusedArgs& a, int f, SeqItem& it, int& c) {
    const VzRagged& r = a.rag;
    const int lane = threadIdx.x % vz::kWave;
    int run = 0;
    for (int s0 = 0; s0 < r.n && run <= a.nc_max; s0 += vz::kWave) {
        const int su = min(s0 + lane, r.n - 1);  // load for every lane, mask after
        const int64_t b = r.base[su];
        const int cp = r.cap[su], ln = r.len[su], np = r.next_pos[su];
        const bool ok = s0 + lane < r.n && vz::decode_status_of(b, cp, ln, np, r.total) == VZ_OK;
        const int n = ok ? (ln + CHUNK) / CHUNK : 0;
        int incl = n;
#pragma unroll
        for (int o = 1; o < vz::kWave; o <<= 1) {
            const int t = __shfl_up(incl, o, vz::kWave);
            if (lane >= o) incl += t;
        }
        const unsigned long long hit = __ballot(run + incl > f);
        if (hit) {
            const int src = __builtin_ctzll(hit);
            const int nc = __builtin_amdgcn_readfirstlane(__shfl(n, src, vz::kWave));
            const int first = __builtin_amdgcn_readfirstlane(run + __shfl(incl, src, vz::kWave) - nc);
            if (first + nc > a.nc_max) return false;
            it.s = s0 + src;
            it.len = __builtin_amdgcn_readfirstlane(__shfl(ln, src, vz::kWave));
            it.next_pos = __builtin_amdgcn_readfirstlane(__shfl(np, src, vz::kWave));
            const uint32_t lo = __builtin_amdgcn_readfirstlane(__shfl(static_cast<int>(b), src, vz::kWave));
            const uint32_t hi = __builtin_amdgcn_readfirstlane(__shfl(static_cast<int>(b >> 32), src, vz::kWave));
            it.base = static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
            it.n_chunks = nc;
            it.first = first;
            c = f - first;
            return true;
        }
        run += __builtin_amdgcn_readfirstlane(__shfl(incl, vz::kWave - 1, vz::kWave));
    }
    return false;
}

// Flat chunk f of a call: false when it holds no work.
template <bool RAG>
__device__ __forceinline__ bool resolve_chunk(const FusedArgs& a, int f, SeqItem& it, int& c) {
    if constexpr (RAG) {
        return locate_ragged_chunk(a, f, it, c);
    } else {
        if (f >= a.n_chunks) return false;
        it.s = 0;
        it.len = a.len;
        it.next_pos = a.next_pos;
        it.n_chunks = a.n_chunks;
        it.first = 0;
        it.base = 0;
        c = f;
    }
    return true;
}

// Attend kernel: work item = (layer, chunk, KV head), a workgroup of SPLIT_W
// waves in which wave w owns keys [VT w, VT w + VT) of the chunk.  Each wave
// requests its query rows and its K and V tile (16 KB) before anything else,
// so a chunk costs one memory round trip, and a one-layer call over 8k keys
// spreads its 16 MB over 260 workgroups.  The waves agree on the chunk's max per head through
// LDS, then sum their exp2 sums and partial outputs in wave order; the
// partial results of (chunk, query head) go to the workspace for the
// finishing kernels.  (Launch bounds: four workgroups per CU, 128 registers
// per lane; the MFMA accumulators then live in ordinary vector registers.)
constexpr int SPLIT_W = CHUNK / VT;  // waves per chunk: one 32-key tile each
template <int NW, bool RAG>
__global__ __launch_bounds__(64 * SPLIT_W, 4) void decode_attend_kernel(const FusedArgs a) {
    constexpr int OS = D + 4;  // padded LDS row of a wave's partial output (floats)
    static_assert(SPLIT_W * GMAX * OS * 4 <= SPLIT_W * TILE_BYTES, "the partial outputs fit in the tile buffers");
    __shared__ __attribute__((aligned(16))) uint8_t s_tile[SPLIT_W][TILE_BYTES];
    __shared__ __attribute__((aligned(16))) uint16_t s_p[GMAX][CHUNK];  // p~ of the chunk, per head
    __shared__ float s_m[SPLIT_W][GMAX], s_l[SPLIT_W][GMAX];
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int q4 = lane >> 4, r16 = lane & 15;
    const int hi = r16 >> 3, hh = r16 & 7;
    const int Hq = a.Hq, nc_max = a.nc_max;
    const int G = Hq / NW;
    // item = (chunk item, KV head), KV head fastest; chunk items are ordered
    // as in the attend kernel (a single sequence's full chunks of every layer
    // first, its short remainders last)
    const int g = static_cast<int>(blockIdx.x) % NW;
    const int ci = static_cast<int>(blockIdx.x) / NW;
    int l, f;
    if constexpr (RAG) {
        l = ci / nc_max;
        f = ci - l * nc_max;
    } else {
        const int n_full = (a.len + 1) / CHUNK;
        if (ci < a.L * n_full) {
            l = ci / n_full;
            f = ci - l * n_full;
        } else {
            l = ci - a.L * n_full;
            f = n_full;
        }
    }
    SeqItem it;
    int c;
    if (!resolve_chunk<RAG>(a, f, it, c)) return;
    const int len = it.len, T = len + 1;
    const int k_begin = chunk_begin(c);
    const int nk = chunk_keys(c, T);
    const int kw0 = k_begin + VT * w;  // the wave's first key
    const int rows = min(VT, max(nk - VT * w, 0));
    const size_t head_base = ((static_cast<size_t>(l) * NW + g) * a.plane + it.base) * D;
    uint16_t* Kh = a.k_cache + head_base;
    uint16_t* Vh = a.v_cache + head_base;
    const size_t row_sl = static_cast<size_t>(it.s) * a.L + l;

    // Eq. (1): the wave whose keys hold slot len (row rr of its tile) loads
    // its KV head's new K and V rows with its other loads, puts them into its
    // tile registers in place of the cache's old row once the tiles have
    // landed, and only then writes them to the cache (and KV head 0 the
    // position), so that none of the chunk's loads waits behind a write.
    // Lane (r16, q4) holds K channels 8 (q4 + 4 s) .. + 7 of its K rows and V
    // channels 8 r16 .. + 7 of its V rows (the tile layouts below).
    const int rr = len - kw0;
    const bool writer = rr >= 0 && rr < VT;  // wave-uniform
    uint4 kn_row[KSTEPS], vn_row;
    if (writer) {
        const uint16_t* kn = a.k_new + (row_sl * NW + g) * D;
        const uint16_t* vn = a.v_new + (row_sl * NW + g) * D;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) kn_row[s] = *reinterpret_cast<const uint4*>(kn + 8 * (q4 + 4 * s));
        vn_row = *reinterpret_cast<const uint4*>(vn + 8 * r16);
    }

    // The query rows first, so that the logits wait for them and the K tile
    // only, not for the V tile behind them.  One descriptor over the KV
    // head's G query rows: lanes of head columns r16 >= G read past it and
    // get zeros, with no memory access.
    uint4 qv[KSTEPS];
    {
        const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t*>(a.q + (row_sl * Hq + g * G) * D), 0, __builtin_amdgcn_readfirstlane(G * D * 2),
            kBufferDword3);
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(rq, (r16 * D + 8 * q4 + 32 * s) * 2, 0, 0);
            __builtin_memcpy(&qv[s], &v, 16);
        }
    }

    // both tiles requested at once; rows past the chunk read as zero without
    // touching memory (bounded scalar descriptors).  The V tile comes whole
    // rows at a time (instruction m: rows 4 m .. 4 m + 3) for its trip through
    // LDS; the K tile straight in the MFMA A-operand layout (register m =
    // 4 ti + s: row 16 ti + r16, bytes 16 (q4 + 4 s) .. + 15), used from
    // registers.
    const int lane_off = q4 * (D * 2) + 16 * r16;
    const int lane_off_k = r16 * (D * 2) + 16 * q4;
    uint4 kt[8], vt[8];
    {
        // (the byte bound taken through readfirstlane keeps the descriptors in
        // scalar registers: a bound left in a vector register makes the
        // compiler wrap every load in a loop over the lanes' descriptors)
        const int nbytes = __builtin_amdgcn_readfirstlane(rows * D * 2);
        const __amdgpu_buffer_rsrc_t rk =
            __builtin_amdgcn_make_buffer_rsrc(Kh + static_cast<size_t>(kw0) * D, 0, nbytes, kBufferDword3);
        const __amdgpu_buffer_rsrc_t rv =
            __builtin_amdgcn_make_buffer_rsrc(Vh + static_cast<size_t>(kw0) * D, 0, nbytes, kBufferDword3);
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(rk, lane_off_k + (m >> 2) * 16 * (D * 2) + (m & 3) * 64,
                                                                 0, 0);
            __builtin_memcpy(&kt[m], &v, 16);
        }
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(rv, lane_off + 4 * m * (D * 2), 0, 0);
            __builtin_memcpy(&vt[m], &v, 16);
        }
    }
    __builtin_amdgcn_sched_barrier(0);  // every load above is issued before the first wait
    uint8_t* const buf = s_tile[w];
    uint8_t* const vwp = buf + q4 * VSTRIDE + 16 * r16;
    const uint8_t* const vr = buf + (4 * q4 + (r16 >> 2)) * VSTRIDE + 16 * ((r16 & 3) >> 1) + 8 * (r16 & 1);

    if (writer && r16 == (rr & 15)) {  // the new K row: row 16 ti + r16 of registers 4 ti .. 4 ti + 3
#pragma unroll
        for (int ti = 0; ti < 2; ++ti)
            if (ti == rr >> 4)
#pragma unroll
                for (int s = 0; s < KSTEPS; ++s) kt[4 * ti + s] = kn_row[s];
    }

    // ---- logits of the wave's 32 keys: S^T = K Q^T ----
    f32x4 acc[2];
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
        acc[ti] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s)
            acc[ti] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kt[4 * ti + s]), as_bf16x8(qv[s]), acc[ti], 0,
                                                              0, 0);
    }
    float sp[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float odd = ror8(acc[1][i]);
        const float v = hi ? odd : acc[0][i];
        const int key = VT * w + 16 * hi + 4 * q4 + i;  // within the chunk
        sp[i] = (key < nk) ? v * a.scale_log2 : -INFINITY;
    }
    float m_w = fmaxf(fmaxf(sp[0], sp[1]), fmaxf(sp[2], sp[3]));
    m_w = fmaxf(m_w, __shfl_xor(m_w, 16, 64));
    m_w = fmaxf(m_w, __shfl_xor(m_w, 32, 64));
    m_w = fmaxf(m_w, ror8(m_w));
    if (q4 == 0 && hi == 0) s_m[w][hh] = m_w;
    if (writer) {
        if (q4 == (rr & 3)) {  // the new V row: row 4 m + q4 of register m
#pragma unroll
            for (int m = 0; m < 8; ++m)
                if (m == rr >> 2) vt[m] = vn_row;
        }
        // the new rows into the cache, after every load of the wave
        if (r16 == (rr & 15)) {
#pragma unroll
            for (int s = 0; s < KSTEPS; ++s) *reinterpret_cast<uint4*>(Kh + len * D + 8 * (q4 + 4 * s)) = kn_row[s];
        }
        if (q4 == (rr & 3)) *reinterpret_cast<uint4*>(Vh + len * D + 8 * r16) = vn_row;
        if (g == 0 && lane == 0) a.pos[static_cast<size_t>(l) * a.plane + it.base + len] = it.next_pos;
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) *reinterpret_cast<uint4*>(vwp + 4 * VSTRIDE * m) = vt[m];
    __syncthreads();

    // ---- the chunk's max per head, p~ against it ----
    float m_c = s_m[0][hh];
#pragma unroll
    for (int v = 1; v < SPLIT_W; ++v) m_c = fmaxf(m_c, s_m[v][hh]);
    float l_w = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        sp[i] = exp2f(sp[i] - m_c);
        l_w += sp[i];
    }
    l_w += __shfl_xor(l_w, 16, 64);
    l_w += __shfl_xor(l_w, 32, 64);
    l_w += ror8(l_w);
    if (q4 == 0 && hi == 0) s_l[w][hh] = l_w;
    const uint32_t p01 = pack_bf16x2(sp[0], sp[1]), p23 = pack_bf16x2(sp[2], sp[3]);
    if (hh < G) *reinterpret_cast<uint2*>(&s_p[hh][VT * w + 16 * hi + 4 * q4]) = make_uint2(p01, p23);

    // ---- O^T = V^T P^T over the wave's keys ----
    float ev[4], od[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float x = sp[i];
        const float y = ror8(x);
        ev[i] = hi ? y : x;
        od[i] = hi ? x : y;
    }
    const uint4 pw = make_uint4(pack_bf16x2(ev[0], ev[1]), pack_bf16x2(ev[2], ev[3]), pack_bf16x2(od[0], od[1]),
                                pack_bf16x2(od[2], od[3]));
    const bf16x8_t pa = as_bf16x8(pw);
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    f32x4 oacc[DTILES];
#pragma unroll
    for (int n = 0; n < DTILES; ++n) {
        s16x4 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(vr + 32 * n));
        s16x4 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)(vr + 16 * VSTRIDE + 32 * n));
        uint4 bw;
        __builtin_memcpy(&bw.x, &b0, 8);
        __builtin_memcpy(&bw.z, &b1, 8);
        oacc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(bw), pa, zero, 0, 0, 0);
    }
    __syncthreads();  // every wave's V reads are done: the tiles take the partial outputs
    float* const s_o = reinterpret_cast<float*>(&s_tile[0][0]);  // [SPLIT_W][GMAX][OS]
    if (r16 < G) {
#pragma unroll
        for (int n = 0; n < DTILES; ++n)
            *reinterpret_cast<f32x4*>(s_o + (w * GMAX + r16) * OS + 16 * n + 4 * q4) = oacc[n];
    }
    __syncthreads();

    // ---- partial results of (chunk, head): (m_c, l_c), O_c and p~ ----
    Partials part(a.ws, a.hdr_bytes, a.L, nc_max, Hq);
    const int pbase = (l * nc_max + it.first + c) * Hq + g * G;  // < 2^31 (checked on the host)
    if (tid < G) {
        float lc = 0.f;
#pragma unroll
        for (int v = 0; v < SPLIT_W; ++v) lc += s_l[v][tid];
        float mc = s_m[0][tid];
#pragma unroll
        for (int v = 1; v < SPLIT_W; ++v) mc = fmaxf(mc, s_m[v][tid]);
        part.ml[pbase + tid] = make_float2(mc, lc);
    }
    {
        // 4 channels (outputs) or 4 keys (p~) per thread, whole rows per head
        const int h = tid >> 5, c4 = 4 * (tid & 31);
        if (h < G) {
            float o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float x = 0.f;
#pragma unroll
                for (int v = 0; v < SPLIT_W; ++v) x += s_o[(v * GMAX + h) * OS + c4 + e];
                o[e] = x;
            }
            *reinterpret_cast<uint2*>(part.o + static_cast<size_t>(pbase + h) * D + c4) =
                make_uint2(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]));
            *reinterpret_cast<uint2*>(part.p + static_cast<size_t>(pbase + h) * CHUNK + c4) =
                *reinterpret_cast<const uint2*>(&s_p[h][c4]);
        }
    }
}

// ---- finishing: merge of the chunk partials ----
// Sums use explicit fused multiply-adds, so the bits do not depend on how the
// compiler contracts each kernel (the single-sequence and ragged calls give
// the same bits).
constexpr int OUT_THREADS = 256;
constexpr int OUT_ROWS = OUT_THREADS / 16;  // row groups
constexpr int OUT_BATCH = 8;                // chunks per row group and round

// Merge of the OUT_ROWS row-group statistics: (layer max M, 1 / sum S).
__device__ __forceinline__ float2 combine_rows(const float* sm, const float* sl, int stride) {
    float Mg = sm[0];
#pragma unroll
    for (int r = 1; r < OUT_ROWS; ++r) Mg = fmaxf(Mg, sm[r * stride]);
    float sum = 0.f;
#pragma unroll
    for (int r = 0; r < OUT_ROWS; ++r) {
        const float f = sm[r * stride] == -INFINITY ? 0.f : exp2f(sm[r * stride] - Mg);
        sum = fmaf(sl[r * stride], f, sum);
    }
    return make_float2(Mg, 1.0f / sum);
}

// One round of a row group's chunks: chunk c0 + OUT_ROWS k of pair st[k] and
// row piece xr[k], while it is below n_chunks, into the running (M, S, acc).
__device__ __forceinline__ void merge_batch(const float2 (&st)[OUT_BATCH], const uint4 (&xr)[OUT_BATCH], int c0,
                                            int n_chunks, float& M, float& S, float (&acc)[8]) {
#pragma unroll
    for (int k = 0; k < OUT_BATCH; ++k) {
        if (c0 + OUT_ROWS * k >= n_chunks) break;
        if (st[k].x > M) {
            const float r = exp2f(M - st[k].x);  // 0 while M is -inf
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] *= r;
            S *= r;
            M = st[k].x;
        }
        const float wgt = exp2f(st[k].x - M);
        float x[8];
        vz::unpack16<VZ_BF16>(xr[k], x);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(wgt, x[i], acc[i]);
        S = fmaf(wgt, st[k].y, S);
    }
}

// The 16 row groups' (M, S, acc) merged in LDS, the output row stored;
// returns the layer's (max, 1 / sum) of head h in thread 0.
__device__ float2 merge_rows_store(const FusedArgs& a, int h, int l, int s, float M, float S, const float (&acc)[8]) {
    __shared__ float s_acc[OUT_ROWS][D + 4];
    __shared__ float s_m[OUT_ROWS], s_l[OUT_ROWS];
    const int t = threadIdx.x, Hq = a.Hq;
    const int rg = t / 16, c8 = 8 * (t % 16);
#pragma unroll
    for (int i = 0; i < 8; ++i) s_acc[rg][c8 + i] = acc[i];
    if (t % 16 == 0) {
        s_m[rg] = M;
        s_l[rg] = S;
    }
    __syncthreads();
    float2 stats = make_float2(0.f, 0.f);
    if (t < D) {
        stats = combine_rows(s_m, s_l, 1);
        float o = 0.f;
#pragma unroll
        for (int r = 0; r < OUT_ROWS; ++r) {
            const float f = s_m[r] == -INFINITY ? 0.f : exp2f(s_m[r] - stats.x);
            o = fmaf(s_acc[r][t], f, o);
        }
        const size_t row_sl = static_cast<size_t>(s) * a.L + l;
        a.out[(row_sl * Hq + h) * D + t] = vz::f32_to_bf16(o * stats.y);
    }
    return stats;
}

// Loads of one round: the pairs and row pieces of chunks c0 + OUT_ROWS k,
// rows clamped to n_load - 1 (every load in bounds, the values masked later).
__device__ __forceinline__ void merge_load(const float2* ml, const uint16_t* po, int Hq, int c0, int n_load,
                                           float2 (&st)[OUT_BATCH], uint4 (&xr)[OUT_BATCH]) {
#pragma unroll
    for (int k = 0; k < OUT_BATCH; ++k) {
        const int cc = min(c0 + OUT_ROWS * k, n_load - 1);
        st[k] = ml[static_cast<size_t>(cc) * Hq];
        xr[k] = *reinterpret_cast<const uint4*>(po + static_cast<size_t>(cc) * Hq * D);
    }
}

// Output row of head h of (layer l, sequence s) from the sequence's n_chunks
// partials starting at chunk row `first`, by a whole block of OUT_THREADS
// threads.  Thread t owns channels 8 (t % 16) .. +7 of the rows of chunks
// t / 16, t / 16 + 16, ...: a running max, o = sum_c O_c exp2(m_c - M) /
// sum_c l_c exp2(m_c - M); the 16 row groups then merge in LDS.  All loads of
// a round (16-byte row pieces and the chunk pairs) are issued before any use:
// indexes past the end are clamped and the values masked afterwards.
// Returns the layer's (max, 1 / sum) of head h in thread 0.
__device__ float2 merge_output_row(const FusedArgs& a, const Partials& part, int h, int l, int s, int first,
                                   int n_chunks) {
    const int t = threadIdx.x, Hq = a.Hq;
    const int rg = t / 16, c8 = 8 * (t % 16);
    const size_t row0 = static_cast<size_t>(l) * a.nc_max + first;  // first chunk row of (layer, sequence)
    const float2* ml = part.ml + row0 * Hq + h;
    const uint16_t* po = part.o + (row0 * Hq + h) * D + c8;
    float M = -INFINITY, S = 0.f, acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
    for (int c0 = rg; c0 < n_chunks; c0 += OUT_ROWS * OUT_BATCH) {
        float2 st[OUT_BATCH];
        uint4 xr[OUT_BATCH];
        merge_load(ml, po, Hq, c0, n_chunks, st, xr);
        merge_batch(st, xr, c0, n_chunks, M, S, acc);
    }
    return merge_rows_store(a, h, l, s, M, S, acc);
}

// Output block of a call of one sequence whose planes hold at most
// OUT_ROWS * OUT_BATCH chunks (one round): its chunk rows start at row 0, so
// the round's loads (rows clamped to the layer's n_load rows) go out before
// the sequence's values arrive, and the same arithmetic as merge_output_row
// follows.  A ragged call of one sequence reports its status here (head 0 of
// layer 0).
template <bool RAG>
__device__ void output_block_one(const FusedArgs& a, int h, int l) {
    const int t = threadIdx.x, Hq = a.Hq;
    const int rg = t / 16, c8 = 8 * (t % 16);
    Partials part(a.ws, a.hdr_bytes, a.L, a.nc_max, Hq);
    const size_t row0 = static_cast<size_t>(l) * a.nc_max;
    float2 st[OUT_BATCH];
    uint4 xr[OUT_BATCH];
    merge_load(part.ml + row0 * Hq + h, part.o + (row0 * Hq + h) * D + c8, Hq, rg, RAG ? a.nc_max : a.n_chunks, st,
               xr);
    int n_chunks = a.n_chunks;
    if constexpr (RAG) {
        const int st0 = vz::ragged_decode_status(a.rag, 0);
        n_chunks = st0 == VZ_OK ? (a.rag.len[0] + CHUNK) / CHUNK : 0;
        const bool ok = st0 == VZ_OK && n_chunks <= a.nc_max;
        if (a.rag.status && h == 0 && l == 0 && t == 0) a.rag.status[0] = ok ? VZ_OK : (st0 != VZ_OK ? st0 : VZ_ERR_CAPACITY);
        if (!ok) return;
    }
    float M = -INFINITY, S = 0.f, acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
    merge_batch(st, xr, rg, n_chunks, M, S, acc);
    merge_rows_store(a, h, l, 0, M, S, acc);
}

// Output kernel, one block per (head, layer, sequence):
// the output row, the layer's (max, 1 / sum) of the head for the fold kernel
// and, in a ragged call, the sequence's status.
template <bool RAG>
__device__ void output_block(const FusedArgs& a, int h, int l, int s_arg, bool store_layer) {
    const int t = threadIdx.x;
    int s = 0, first = 0, n_chunks = a.n_chunks;
    if constexpr (RAG) {
        s = s_arg;
        // the sequence's own values and the earlier sequences' chunk counts
        // are loaded side by side (one round of loads)
        const int st = vz::ragged_decode_status(a.rag, s);
        const int fst = vz::ragged_first(s, a.nc_max, [&](int u) { return ragged_chunks(a.rag, u); });
        first = st == VZ_OK ? fst : -1;
        n_chunks = st == VZ_OK ? (a.rag.len[s] + CHUNK) / CHUNK : 0;
        const bool ok = st == VZ_OK && first >= 0 && first + n_chunks <= a.nc_max;
        if (a.rag.status && h == 0 && l == 0 && t == 0) a.rag.status[s] = ok ? VZ_OK : (st != VZ_OK ? st : VZ_ERR_CAPACITY);
        if (!ok) return;
    }
    Partials part(a.ws, a.hdr_bytes, a.L, a.nc_max, a.Hq);
    const float2 stats = merge_output_row(a, part, h, l, s, first, n_chunks);
    if (store_layer && t == 0) part.layer[(static_cast<size_t>(s) * a.L + l) * a.Hq + h] = stats;
}

template <bool RAG>
__global__ __launch_bounds__(OUT_THREADS) void decode_output_kernel(const FusedArgs a) {
    output_block<RAG>(a, blockIdx.x, blockIdx.y, blockIdx.z, true);
}

// Fold kernel, one block of CHUNK threads per (chunk, layer), thread = key:
// Eq. (6), A[j] = gamma A[j] + sum_h p~_hj f_h with f_h = exp2(m_c,h - M_h) / S_h
// from the layer statistics the output kernel stored (the new slot starts
// from 0).  Heads go in rounds of 32: the round's p~ loads are issued before
// its factors are formed (p~ rows are complete, CHUNK entries each, so every
// load is in bounds; heads past Hq are clamped and masked, so no load sits
// behind a branch).
constexpr int FOLD_HEADS = 32;
template <bool RAG>
__global__ __launch_bounds__(CHUNK) void decode_fold_kernel(const FusedArgs a) {
    __shared__ float s_f[FOLD_HEADS];
    const int l = blockIdx.y, t = threadIdx.x;
    const int Hq = a.Hq;
    SeqItem it;
    int c;
    if (!resolve_chunk<RAG>(a, blockIdx.x, it, c)) return;
    const ConstPartials part(a.ws, a.hdr_bytes, a.L, a.nc_max, Hq);
    const int len = it.len, T = len + 1;
    const int k_begin = chunk_begin(c);
    const int nk = chunk_keys(c, T);
    const int j = k_begin + (t < nk ? t : 0);
    float* sc = a.score + static_cast<size_t>(l) * a.plane + it.base + j;
    const float a_ld = *sc;
    const float a_old = (t < nk && j < len) ? a_ld : 0.f;  // zero pad of Eq. (6) for the new slot
    const size_t cbase = (static_cast<size_t>(l) * a.nc_max + it.first + c) * Hq;
    const float2* layer = part.layer + (static_cast<size_t>(it.s) * a.L + l) * Hq;
    const uint16_t* pp = part.p + cbase * CHUNK + t;
    float acc = 0.f;
    for (int hb = 0; hb < Hq; hb += FOLD_HEADS) {
        uint16_t pr[FOLD_HEADS];
#pragma unroll
        for (int q = 0; q < FOLD_HEADS; ++q) pr[q] = pp[min(hb + q, Hq - 1) * CHUNK];
        if (t < FOLD_HEADS && hb + t < Hq) {
            const float2 gl = layer[hb + t];
            s_f[t] = exp2f(part.ml[cbase + hb + t].x - gl.x) * gl.y;
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < FOLD_HEADS; ++q)
            if (hb + q < Hq) acc = fmaf(vz::bf16_to_f32(pr[q]), s_f[q], acc);
        __syncthreads();
    }
    if (t < nk) *sc = fmaf(a.gamma, a_old, acc);
}

// Output merge and score fold in one launch, for calls whose sequences have
// few chunks (planes of at most FINISH_MAX_CHUNKS chunks).  Blocks
// [0, n_chunks) of a layer are fold blocks: one per chunk, each forms every
// head's layer statistics itself from its sequence's chunk pairs, with the
// output kernel's arithmetic and order (the same bits), then folds its
// chunk's keys as the fold kernel does.  The blocks after them are the output
// kernel's blocks, one per (head, sequence), run beside the fold blocks.  The
// recomputation reads n_chunks x Hq pairs per fold block, cheap while chunks
// are few.
constexpr int FINISH_MAX_CHUNKS = 128;
constexpr int FINISH_MAX_HEADS = 8 * GMAX;  // Hq <= Hkv * GMAX with Hkv <= 8
template <bool RAG>
__global__ __launch_bounds__(OUT_THREADS) void decode_finish_kernel(const FusedArgs a) {
    __shared__ float s_gm[FINISH_MAX_HEADS * OUT_ROWS], s_gl[FINISH_MAX_HEADS * OUT_ROWS];
    __shared__ float2 s_stat[FINISH_MAX_HEADS];
    __shared__ float s_f[FOLD_HEADS];
    const int t = threadIdx.x, l = blockIdx.y, Hq = a.Hq;
    // One sequence (a single-sequence call, or a ragged call of one): its
    // chunk rows start at row 0 of the layer and a fold block's chunk is row
    // blockIdx.x, so every partial-result load is issued before the
    // sequence's values are known (rows clamped to the layer's rows, values
    // masked once they are): one round of loads instead of two.
    const bool one = !RAG || a.rag.n == 1;
    if (static_cast<int>(blockIdx.x) >= a.n_chunks) {
        const int ob = static_cast<int>(blockIdx.x) - a.n_chunks;
        if (one)
            output_block_one<RAG>(a, ob % Hq, l);
        else
            output_block<RAG>(a, ob % Hq, l, ob / Hq, false);
        return;
    }
    const ConstPartials part(a.ws, a.hdr_bytes, a.L, a.nc_max, Hq);
    // Loads first, all independent of one another: the chunk pairs of the
    // statistics (thread t: (head, row group) pairs t, t + OUT_THREADS, ...,
    // up to FINISH_GROUP_CHUNKS chunks each, indexes clamped), the fold's p~
    // of the first FOLD_HEADS heads, its chunk's own pairs and the scores.
    constexpr int FINISH_GROUP_CHUNKS = FINISH_MAX_CHUNKS / OUT_ROWS;
    constexpr int FINISH_PAIRS = FINISH_MAX_HEADS * OUT_ROWS / OUT_THREADS;
    float2 stv[FINISH_PAIRS][FINISH_GROUP_CHUNKS];
    uint16_t pr[FOLD_HEADS];
    float m_own;
    const int tk = t < CHUNK ? t : 0;
    // (head, row group) pair pi = rg * Hq + h: the 64 lanes of a load
    // instruction read whole rows of heads (two rows of 32 heads, four cache
    // lines); rounds past the Hq * OUT_ROWS pairs are skipped (uniform)
    auto load_pairs = [&](size_t row0, int n_load) {
#pragma unroll
        for (int u = 0; u < FINISH_PAIRS; ++u) {
            if (u * OUT_THREADS >= Hq * OUT_ROWS) break;
            const int pi = min(t + u * OUT_THREADS, Hq * OUT_ROWS - 1);
            const int rg = pi / Hq, h = pi - rg * Hq;
#pragma unroll
            for (int k = 0; k < FINISH_GROUP_CHUNKS; ++k)
                stv[u][k] = part.ml[(row0 + min(rg + k * OUT_ROWS, n_load - 1)) * Hq + h];
        }
    };
    auto load_own = [&](size_t cbase) {
        const uint16_t* pp = part.p + cbase * CHUNK + tk;
#pragma unroll
        for (int q = 0; q < FOLD_HEADS; ++q) pr[q] = pp[min(q, Hq - 1) * CHUNK];
        m_own = part.ml[cbase + min(t % FOLD_HEADS, Hq - 1)].x;
    };
    SeqItem it;
    int c;
    float a_spec = 0.f;
    if (one) {
        // the sequence's values first (a ragged call of one: sequence 0 owns
        // chunk rows [0, its chunks)), then the partial results, then the
        // checks: the score load below waits only for the values
        int64_t b = 0;
        int cp = a.plane, ln = a.len, np = a.next_pos;
        if constexpr (RAG) {
            b = a.rag.base[0];
            cp = a.rag.cap[0];
            ln = a.rag.len[0];
            np = a.rag.next_pos[0];
        }
        load_pairs(static_cast<size_t>(l) * a.nc_max, RAG ? a.nc_max : a.n_chunks);
        load_own((static_cast<size_t>(l) * a.nc_max + blockIdx.x) * Hq);
        // the score of key tk of chunk blockIdx.x for a sequence at slot 0
        // (a single-sequence call, or the one slot of a decode loop), with the
        // other loads; another base loads it again once the values are in
        a_spec = a.score[static_cast<size_t>(l) * a.plane +
                         min(static_cast<int64_t>(chunk_begin(blockIdx.x) + tk), a.plane - 1)];
        int nc = a.n_chunks;
        if constexpr (RAG) {
            const bool ok = vz::decode_status_of(b, cp, ln, np, a.rag.total) == VZ_OK;
            nc = ok ? (ln + CHUNK) / CHUNK : 0;
            if (nc > a.nc_max) nc = 0;
        }
        if (static_cast<int>(blockIdx.x) >= nc) return;
        it.s = 0;
        it.len = ln;
        it.next_pos = np;
        it.n_chunks = nc;
        it.first = 0;
        it.base = b;
        c = blockIdx.x;
    } else if (!resolve_chunk<RAG>(a, blockIdx.x, it, c)) {
        return;
    }
    const size_t row0 = static_cast<size_t>(l) * a.nc_max + it.first;
    const int nch = it.n_chunks;
    const size_t cbase = (row0 + c) * Hq;  // = (layer row + blockIdx.x) * Hq
    if (!one) {
        load_pairs(row0, nch);
        load_own(cbase);
    }
    const int len = it.len, T = len + 1;
    const int nk = chunk_keys(c, T);
    const int j = chunk_begin(c) + (tk < nk ? tk : 0);
    float* sc = a.score + static_cast<size_t>(l) * a.plane + it.base + j;
    // (used only for tk < nk, where j is the slot the speculative load read)
    const float a_ld = one && it.base == 0 ? a_spec : *sc;
    const uint16_t* pp = part.p + cbase * CHUNK + tk;

    // the layer statistics of every head: row group rg of head h takes
    // chunks rg, rg + OUT_ROWS, ... with a running max, then the groups merge
#pragma unroll
    for (int u = 0; u < FINISH_PAIRS; ++u) {
        const int pi = t + u * OUT_THREADS;
        if (pi < Hq * OUT_ROWS) {
            const int rg = pi / Hq, h = pi - rg * Hq;
            float M = -INFINITY, S = 0.f;
#pragma unroll
            for (int k = 0; k < FINISH_GROUP_CHUNKS; ++k) {
                if (rg + k * OUT_ROWS >= nch) break;
                const float2 st = stv[u][k];
                if (st.x > M) {
                    S *= exp2f(M - st.x);
                    M = st.x;
                }
                S = fmaf(exp2f(st.x - M), st.y, S);
            }
            s_gm[h * OUT_ROWS + rg] = M;
            s_gl[h * OUT_ROWS + rg] = S;
        }
    }
    __syncthreads();
    if (t < Hq) s_stat[t] = combine_rows(&s_gm[t * OUT_ROWS], &s_gl[t * OUT_ROWS], 1);
    __syncthreads();

    // Eq. (6) for the chunk's keys (threads below CHUNK), as the fold kernel
    const float a_old = (tk < nk && j < len) ? a_ld : 0.f;
    float acc = 0.f;
    for (int hb = 0; hb < Hq; hb += FOLD_HEADS) {
        if (hb > 0) {
#pragma unroll
            for (int q = 0; q < FOLD_HEADS; ++q) pr[q] = pp[min(hb + q, Hq - 1) * CHUNK];
        }
        if (t < FOLD_HEADS && hb + t < Hq) {
            const float2 gl = s_stat[hb + t];
            const float m_c = hb == 0 ? m_own : part.ml[cbase + hb + t].x;
            s_f[t] = exp2f(m_c - gl.x) * gl.y;
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < FOLD_HEADS; ++q)
            if (hb + q < Hq) acc = fmaf(vz::bf16_to_f32(pr[q]), s_f[q], acc);
        __syncthreads();
    }
    if (t < CHUNK && t < nk) *sc = fmaf(a.gamma, a_old, acc);
}

// Chunk rows of the partials per layer: ceil(plane / CHUNK) for a single
// sequence; for a ragged call ceil(plane / CHUNK) + n_seqs, a bound on the
// sum of ceil((len[s] + 1) / CHUNK) over sequences that lie inside the planes
// without overlapping.
int64_t chunk_rows(int64_t plane, int32_t n_seqs) {
    return (plane + CHUNK - 1) / CHUNK + (n_seqs > 0 ? n_seqs : 0);
}

template <int NW, bool RAG>
hipError_t launch_decode_fused(const VzDecodeArgs& v, hipStream_t stream) {
    FusedArgs a{};
    a.q = static_cast<const uint16_t*>(v.q);
    a.k_new = static_cast<const uint16_t*>(v.k_new);
    a.v_new = static_cast<const uint16_t*>(v.v_new);
    a.k_cache = static_cast<uint16_t*>(v.k_cache);
    a.v_cache = static_cast<uint16_t*>(v.v_cache);
    a.pos = v.pos;
    a.score = v.score;
    a.out = static_cast<uint16_t*>(v.out);
    a.ws = static_cast<uint8_t*>(v.ws);
    a.Hq = v.Hq;
    a.L = v.L;
    a.hdr_bytes = static_cast<int32_t>(vz_decode_hdr_bytes(v.L));
    a.scale_log2 = (v.sm_scale > 0.f ? v.sm_scale : 1.0f / sqrtf(static_cast<float>(D))) * kLog2e;
    a.gamma = v.gamma;
    a.rag = v.rag;
    int seqs = 1;
    if (RAG) {
        a.plane = v.rag.total;
        a.nc_max = static_cast<int32_t>(chunk_rows(a.plane, v.rag.n));
        a.n_chunks = a.nc_max;  // grid extent per layer
        seqs = v.rag.n;
    } else {
        a.plane = v.cap;
        a.len = v.len;
        a.next_pos = v.next_pos;
        a.n_chunks = static_cast<int32_t>((static_cast<int64_t>(v.len) + CHUNK) / CHUNK);  // of len + 1 keys
        a.nc_max = static_cast<int32_t>(chunk_rows(a.plane, 0));
    }
    if (vz_decode_range_ok(a.L, NW, RAG ? v.rag.n : 0)) {
        if (!RAG) {
            a.cnt = reinterpret_cast<uint64_t*>(a.ws + kHeaderBytes);
            a.tag = vz_call_tag();
            a.ev = v.ev;
            a.ev_budget = v.ev_budget;
            a.ev_sink = v.ev_sink;
            a.ev_M = v.ev_M;
            a.ev_kept = v.ev_kept;
            a.ev_n = v.ev_n;
        }
        return vz_launch_decode_range(a, NW, stream);
    }
    hipLaunchKernelGGL((decode_attend_kernel<NW, RAG>), dim3(a.L * a.n_chunks * NW), dim3(64 * SPLIT_W), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((a.plane + CHUNK - 1) / CHUNK <= FINISH_MAX_CHUNKS) {
        hipLaunchKernelGGL((decode_finish_kernel<RAG>), dim3(a.n_chunks + a.Hq * seqs, a.L), dim3(OUT_THREADS), 0,
                           stream, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((decode_output_kernel<RAG>), dim3(a.Hq, a.L, seqs), dim3(OUT_THREADS), 0, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((decode_fold_kernel<RAG>), dim3(a.n_chunks, a.L), dim3(CHUNK), 0, stream, a);
    return hipGetLastError();
}

template <int NW>
hipError_t launch_decode_fused_any(const VzDecodeArgs& v, hipStream_t stream) {
    return v.rag.n > 0 ? launch_decode_fused<NW, true>(v, stream) : launch_decode_fused<NW, false>(v, stream);
}

}  // namespace

// ---- sizing shared with the host API ----
size_t vz_decode_hdr_bytes(int32_t L) {
    return kHeaderBytes + (static_cast<size_t>(L) * sizeof(uint64_t) + 255) / 256 * 256;
}

uint32_t vz_call_tag() {
    static std::atomic<uint32_t> next{static_cast<uint32_t>(std::random_device{}())};
    uint32_t t;
    do t = next.fetch_add(1, std::memory_order_relaxed);
    while (t == 0);
    return t;
}

bool vz_decode_fused_ok(int32_t dtype, int32_t d, int32_t Hq, int32_t Hkv, int32_t L, int64_t plane, int32_t n_seqs) {
    if (dtype != VZ_BF16 || d != D) return false;
    if (!(Hkv == 1 || Hkv == 2 || Hkv == 4 || Hkv == 8)) return false;
    if (Hq % Hkv != 0 || Hq / Hkv > GMAX) return false;
    // 32-bit chunk-row indexes of the partials (the attend grid is smaller)
    return static_cast<int64_t>(L) * chunk_rows(plane, n_seqs) * Hq < (int64_t(1) << 31);
}

size_t vz_decode_fused_ws_bytes(int32_t L, int32_t Hq, int64_t plane, int32_t n_seqs) {
    const int64_t rows = chunk_rows(plane, n_seqs);
    const int32_t seqs = n_seqs > 0 ? n_seqs : 1;
    return vz_decode_hdr_bytes(L) + static_cast<size_t>(L) * rows * Hq * (sizeof(float2) + sizeof(uint16_t) * (D + CHUNK)) +
           static_cast<size_t>(seqs) * L * Hq * sizeof(float2);
}

hipError_t vz_launch_decode_fused(const VzDecodeArgs& a, hipStream_t stream) {
    switch (a.Hkv) {
        case 1: return launch_decode_fused_any<1>(a, stream);
        case 2: return launch_decode_fused_any<2>(a, stream);
        case 4: return launch_decode_fused_any<4>(a, stream);
        case 8: return launch_decode_fused_any<8>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

bool vz_decode_takes_range(const VzDecodeArgs& a) {
    return a.rag.n == 0 && vz_decode_fused_ok(a.dtype, a.d, a.Hq, a.Hkv, a.L, a.cap, 0) &&
           vz_decode_range_ok(a.L, a.Hkv, 0) && vz_decode_range_whole(a.len);
}

bool vz_decode_evicts(const VzDecodeArgs& a, int32_t budget) {
    const int64_t T = static_cast<int64_t>(a.len) + 1;
    const int64_t E = T > budget ? T - budget : 0;
    return vz_decode_takes_range(a) && a.Hkv <= 4 && E <= vz_sel::kInlineRows;
}
