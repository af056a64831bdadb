// Decode step (Sec. 3.1 Eq. 1-2, Sec. 3.2.2 Eq. 6) for bfloat16 caches with
// d = 128 and at most 8 query heads per KV head, chunked path.  Three
// launches cover every layer: the attend kernel streams the cache once and
// leaves per-chunk partial results in the workspace; the output and fold
// kernels merge them into the output rows and the decayed scores.  No
// workgroup ever waits for another.  Single-sequence calls with enough
// (layer, KV head) items and a short enough cache go to the whole-range path
// (decode_range.hip) instead.
//
// Attend kernel: work item = (layer, key chunk of <= 128 keys).  A workgroup
// has one wave per KV head; wave g streams K and V rows of head g over the
// chunk.  Registers stay under 128 per lane so that four workgroups share a
// CU.
//   pass 1  S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (M = 16 keys, N = 16
//           query-head columns of which n_q/n_kv <= 8 are used, K = 32
//           channels).  K tiles of 32 rows are loaded fully coalesced (4 whole
//           rows per 1 KB instruction), stored to LDS with padded rows and
//           read back with ds_read_b128 in the A-operand layout.  One tile is
//           in flight while the previous one is multiplied; the first V tile
//           follows the last K tile.  The logits of an odd 16-key tile are
//           moved into the unused head columns 8..15 of the even tile's
//           registers (DPP row rotate by 8), so 128 keys x 8 heads take 16
//           registers per lane.
//   stats   chunk-local max m_c and sum l_c of exp2 per head; the registers
//           then hold p~ = exp2(s - m_c).  (m_c, l_c) and p~ (bfloat16,
//           64 bytes per key over the 32 heads of the workload) go to the
//           workspace.
//   pass 2  O_c = P V: V tiles take the same coalesced path into LDS and are
//           read back with ds_read_b64_tr_b16 directly in the B-operand
//           layout; P is rebuilt from the packed p~ registers with one row
//           rotate.  O_c (relative to m_c) goes to the workspace in bfloat16.
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

constexpr int ATTEND_WG_PER_CU = 4;  // resident attend workgroups per CU (128 VGPRs)
constexpr int ATTEND_DEEP_MAX_ITEMS = 512;  // attend grids this small keep four tiles in flight per wave
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

// Flat chunk f of a call: false when it holds no work.
template <bool RAG>
__device__ __forceinline__ bool resolve_chunk(const FusedArgs& a, int f, SeqItem& it, int& c) {
    if constexpr (RAG) {
        int first = 0, nc = 0;
        const int s = vz::ragged_locate(f, a.rag.n, a.nc_max, [&](int t) { return ragged_chunks(a.rag, t); },
                                        first, nc);
        if (s < 0 || first + nc > a.nc_max) return false;
        it.s = s;
        it.len = __builtin_amdgcn_readfirstlane(a.rag.len[s]);
        it.next_pos = __builtin_amdgcn_readfirstlane(a.rag.next_pos[s]);
        it.n_chunks = nc;
        it.first = first;
        it.base = a.rag.base[s];
        c = f - first;
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

// DEPTH: K/V tiles in flight per wave.  1 keeps the registers within four
// resident workgroups per CU; 4 (the K tiles at once, each V tile issued as
// its K slot frees) shortens the chain of dependent loads for grids too small
// to fill the GPU, where occupancy does not matter.  The arithmetic is the
// same, so are the bits.
template <int NW, bool RAG, int DEPTH>
__global__ __launch_bounds__(64 * NW, DEPTH == 1 ? ATTEND_WG_PER_CU : 1) void decode_attend_kernel(const FusedArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t s_tile[NW][TILE_BYTES];
    const int tid = threadIdx.x;
    // wave-uniform values go through readfirstlane so that addresses built
    // from them stay scalar (buffer descriptors in SGPRs)
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int q4 = lane >> 4, r16 = lane & 15;
    const int hi = r16 >> 3;          // 0: even tile of a pair, 1: odd tile (packed lanes)
    const int hh = r16 & 7;           // query head of the group this lane's logits belong to
    const int Hq = a.Hq, nc_max = a.nc_max;
    const int G = Hq / NW;
    const int g = w;                  // KV head of this wave

    Partials part(a.ws, a.hdr_bytes, a.L, nc_max, Hq);
    // Work order: a single sequence's full chunks of every layer come first
    // and the layers' short remainder chunks last, so the partial last round
    // of workgroups is the cheap one.  A ragged call goes layer by layer.
    const int item = blockIdx.x;
    int l, f;
    if constexpr (RAG) {
        l = item / nc_max;
        f = item - l * nc_max;
    } else {
        const int n_full = (a.len + 1) / CHUNK;
        if (item < a.L * n_full) {
            l = item / n_full;
            f = item - l * n_full;
        } else {
            l = item - a.L * n_full;
            f = n_full;
        }
    }
    SeqItem it;
    int c;
    if (!resolve_chunk<RAG>(a, f, it, c)) return;
    const int len = it.len;
    const int T = len + 1;
    const int k_begin = chunk_begin(c);
    const int nk = chunk_keys(c, T);
    const size_t head_base = ((static_cast<size_t>(l) * NW + g) * a.plane + it.base) * D;
    uint16_t* Kh = a.k_cache + head_base;
    uint16_t* Vh = a.v_cache + head_base;
    const size_t row_sl = static_cast<size_t>(it.s) * a.L + l;  // (sequence, layer) row of q, out, k_new, v_new

    // Eq. (1) first: the chunk holding slot len writes the new row into the
    // cache (the wave of each KV head its own row, complete before its loads),
    // so every key is read from the cache the same way.
    if (len >= k_begin && len < k_begin + nk) {
        const uint16_t* kn = a.k_new + (row_sl * NW + g) * D;
        const uint16_t* vn = a.v_new + (row_sl * NW + g) * D;
        if (lane < 16)
            *reinterpret_cast<uint4*>(Kh + len * D + 8 * lane) = *reinterpret_cast<const uint4*>(kn + 8 * lane);
        else if (lane < 32)
            *reinterpret_cast<uint4*>(Vh + len * D + 8 * (lane - 16)) =
                *reinterpret_cast<const uint4*>(vn + 8 * (lane - 16));
        if (tid == 0) a.pos[static_cast<size_t>(l) * a.plane + it.base + len] = it.next_pos;
        __threadfence_block();
    }

    // Staging: the chunk's K rows and then its V rows stream through the
    // registers as one sequence of 8 tiles of 32 rows.  Instruction m of a
    // tile reads rows 4m..4m+3 whole (lane = row 4m + q4, 16-byte column r16)
    // with buffer loads from a descriptor based at the tile's first row and
    // bounded to the chunk's rows, so rows past the chunk end read as zero and
    // cost no memory traffic (their logits are masked, their probabilities
    // are zero).  The descriptor is scalar; every load shares the lane offset.
    const uint16_t* const kc = Kh + static_cast<size_t>(k_begin) * D;
    const uint16_t* const vc = Vh + static_cast<size_t>(k_begin) * D;
    const int lane_off = q4 * (D * 2) + 16 * r16;
    // tile tt: K tiles 0 .. PAIRS - 1, then V tiles; held in slot tt % DEPTH
    uint4 stg[DEPTH][8];
    auto load_tile = [&](int tt) {
        const uint16_t* base = tt < PAIRS ? kc : vc;
        const int u = tt % PAIRS;
        const int rows = nk - VT * u > 0 ? nk - VT * u : 0;
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base) + VT * u * D, 0, rows * D * 2, kBufferDword3);
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, lane_off + 4 * m * (D * 2), 0, 0);
            __builtin_memcpy(&stg[tt % DEPTH][m], &v, 16);
        }
    };
#pragma unroll
    for (int tt = 0; tt < DEPTH; ++tt) load_tile(tt);

    // Per-lane LDS bases.  Stores: lane (q4, r16) writes 16-byte column r16 of
    // row 4m + q4 in instruction m.  K reads (A operand of S^T = K Q^T): row
    // r16 (+16 for the odd tile), columns 4s + q4.  V reads (transposed B
    // operand of P V): in each 16-lane group, row 4 q4 + r16 / 4 (+16 for
    // keys 16..31 of the tile), 8 bytes at column 32 n + 16 ((r16 & 3) / 2) +
    // 8 (r16 & 1).
    uint8_t* const buf = s_tile[w];
    uint8_t* const kw = buf + q4 * KSTRIDE + 16 * r16;
    uint8_t* const vw = buf + q4 * VSTRIDE + 16 * r16;
    const uint8_t* const kr = buf + r16 * KSTRIDE + 16 * q4;
    const uint8_t* const vr = buf + (4 * q4 + (r16 >> 2)) * VSTRIDE + 16 * ((r16 & 3) >> 1) + 8 * (r16 & 1);

    // ---------------- pass 1: logits S^T = K Q^T ----------------
    uint4 qv[KSTEPS];  // B operand: Q^T, column r16 = query head (zero past G)
    {
        const int hq = r16 < G ? r16 : 0;
        const uint16_t* qrow = a.q + (row_sl * Hq + g * G + hq) * D + 8 * q4;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
            const uint4 v = *reinterpret_cast<const uint4*>(qrow + 32 * s);
            qv[s] = (r16 < G) ? v : make_uint4(0, 0, 0, 0);
        }
    }
    // sp[u][i]: lanes with hi = 0 hold key 32u + 4 q4 + i, head hh; lanes with
    // hi = 1 hold key 32u + 16 + 4 q4 + i, head hh.
    float sp[PAIRS][4];
#pragma unroll
    for (int u = 0; u < PAIRS; ++u) {
#pragma unroll
        for (int m = 0; m < 8; ++m) *reinterpret_cast<uint4*>(kw + 4 * KSTRIDE * m) = stg[u % DEPTH][m];
        if (u + DEPTH < 2 * PAIRS) load_tile(u + DEPTH);  // the V tiles follow the K tiles
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the tile is in LDS
        f32x4 acc[2];
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) {
            acc[ti] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < KSTEPS; ++s) {
                const uint4 a = *reinterpret_cast<const uint4*>(kr + 16 * KSTRIDE * ti + 64 * s);
                acc[ti] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(qv[s]), acc[ti], 0, 0, 0);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float odd = ror8(acc[1][i]);  // lane hi=1 receives the odd tile of head hh
            const float v = hi ? odd : acc[0][i];
            const int key = VT * u + 16 * hi + 4 * q4 + i;
            sp[u][i] = (key < nk) ? v * a.scale_log2 : -INFINITY;
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the next tile is stored
    }

    // ---------------- chunk statistics ----------------
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
    const int pbase = (l * nc_max + it.first + c) * Hq + g * G;  // < 2^31 (checked on the host)
    if (q4 == 0 && r16 < G) part.ml[pbase + r16] = make_float2(m_c, l_c);

    // ---------------- pass 2: O^T = V^T P^T on the matrix cores ----------------
    // (D tile n: column = head r16, rows = channels 16 n + 4 q4 + 0..3, so each
    // lane ends with runs of 4 channels of one head)
    f32x4 oacc[DTILES];
#pragma unroll
    for (int n = 0; n < DTILES; ++n) oacc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < PAIRS; ++u) {
#pragma unroll
        for (int m = 0; m < 8; ++m) *reinterpret_cast<uint4*>(vw + 4 * VSTRIDE * m) = stg[(PAIRS + u) % DEPTH][m];
        if (PAIRS + u + DEPTH < 2 * PAIRS) load_tile(PAIRS + u + DEPTH);
        // B operand P^T: column = head r16 (columns >= G feed output columns
        // that are never stored), k-slots 8 q4 + i -> keys 32u + 4 q4 + i (i < 4)
        // and 32u + 16 + 4 q4 + i - 4 (i >= 4): the even tile is in place, the
        // odd tile comes back from the upper half of the row.
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
    // ---------------- partial results: whole rows through LDS ----------------
    // p~ (bfloat16, CHUNK entries per head) and O (bfloat16 relative to the chunk
    // max, 256 bytes per head) of the wave's G heads are staged in its free
    // tile buffer at padded per-head strides, then written as 1 KB fully
    // coalesced stores: the workspace holds both as rows, heads of the wave
    // adjacent.
    {
        constexpr int PR = CHUNK * 2, HSP = PR + 64, HS = 256 + 64;
        static_assert(GMAX * (HSP + HS) <= TILE_BYTES, "the staged partials fit in the tile buffer");
        uint8_t* const lp = buf;
        uint8_t* const lo = buf + GMAX * HSP;
        if (hh < G) {
#pragma unroll
            for (int u = 0; u < PAIRS; ++u)
                *reinterpret_cast<uint2*>(lp + hh * HSP + 2 * (VT * u + 16 * hi + 4 * q4)) =
                    make_uint2(pack_bf16x2(sp[u][0], sp[u][1]), pack_bf16x2(sp[u][2], sp[u][3]));
        }
        if (r16 < G) {
#pragma unroll
            for (int n = 0; n < DTILES; ++n)
                *reinterpret_cast<uint2*>(lo + r16 * HS + 2 * (16 * n + 4 * q4)) =
                    make_uint2(pack_bf16x2(oacc[n][0], oacc[n][1]), pack_bf16x2(oacc[n][2], oacc[n][3]));
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): staged
        uint8_t* const gp = reinterpret_cast<uint8_t*>(part.p) + static_cast<size_t>(pbase) * PR;
        uint8_t* const go = reinterpret_cast<uint8_t*>(part.o) + static_cast<size_t>(pbase) * (D * 2);
#pragma unroll
        for (int j = 0; j < GMAX * PR / 1024; ++j) {
            const int off = 1024 * j + 16 * lane;
            if (off < G * PR)
                *reinterpret_cast<uint4*>(gp + off) =
                    *reinterpret_cast<const uint4*>(lp + (off / PR) * HSP + off % PR);
        }
#pragma unroll
        for (int j = 0; j < GMAX * 256 / 1024; ++j) {
            const int off = 1024 * j + 16 * lane;
            if (off < G * 256)
                *reinterpret_cast<uint4*>(go + off) = *reinterpret_cast<const uint4*>(lo + (off >> 8) * HS + (off & 255));
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
    __shared__ float s_acc[OUT_ROWS][D + 4];
    __shared__ float s_m[OUT_ROWS], s_l[OUT_ROWS];
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
#pragma unroll
        for (int k = 0; k < OUT_BATCH; ++k) {
            const int cc = min(c0 + OUT_ROWS * k, n_chunks - 1);
            st[k] = ml[static_cast<size_t>(cc) * Hq];
            xr[k] = *reinterpret_cast<const uint4*>(po + static_cast<size_t>(cc) * Hq * D);
        }
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

// Output kernel, one block per (head, layer, sequence):
// the output row, the layer's (max, 1 / sum) of the head for the fold kernel
// and, in a ragged call, the sequence's status.
template <bool RAG>
__device__ void output_block(const FusedArgs& a, int h, int l, int s_arg, bool store_layer) {
    const int t = threadIdx.x;
    int s = 0, first = 0, n_chunks = a.n_chunks;
    if constexpr (RAG) {
        s = s_arg;
        const int st = vz::ragged_decode_status(a.rag, s);
        first = st == VZ_OK ? vz::ragged_first(s, a.nc_max, [&](int u) { return ragged_chunks(a.rag, u); }) : -1;
        n_chunks = st == VZ_OK ? ragged_chunks(a.rag, s) : 0;
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
    if (static_cast<int>(blockIdx.x) >= a.n_chunks) {
        const int ob = static_cast<int>(blockIdx.x) - a.n_chunks;
        output_block<RAG>(a, ob % Hq, l, ob / Hq, false);
        return;
    }
    SeqItem it;
    int c;
    if (!resolve_chunk<RAG>(a, blockIdx.x, it, c)) return;
    const ConstPartials part(a.ws, a.hdr_bytes, a.L, a.nc_max, Hq);
    const size_t row0 = static_cast<size_t>(l) * a.nc_max + it.first;
    const int nch = it.n_chunks;
    // Loads first, all independent of one another: the chunk pairs of the
    // statistics (thread t: (head, row group) pairs t, t + OUT_THREADS, ...,
    // up to FINISH_GROUP_CHUNKS chunks each, indexes clamped), the fold's p~
    // of the first FOLD_HEADS heads, its chunk's own pairs and the scores.
    constexpr int FINISH_GROUP_CHUNKS = FINISH_MAX_CHUNKS / OUT_ROWS;
    constexpr int FINISH_PAIRS = FINISH_MAX_HEADS * OUT_ROWS / OUT_THREADS;
    float2 stv[FINISH_PAIRS][FINISH_GROUP_CHUNKS];
#pragma unroll
    for (int u = 0; u < FINISH_PAIRS; ++u) {
        const int pi = min(t + u * OUT_THREADS, Hq * OUT_ROWS - 1);
        const int h = pi / OUT_ROWS, rg = pi - h * OUT_ROWS;
#pragma unroll
        for (int k = 0; k < FINISH_GROUP_CHUNKS; ++k)
            stv[u][k] = part.ml[(row0 + min(rg + k * OUT_ROWS, nch - 1)) * Hq + h];
    }
    const int len = it.len, T = len + 1;
    const int nk = chunk_keys(c, T);
    const int tk = t < CHUNK ? t : 0;
    const int j = chunk_begin(c) + (tk < nk ? tk : 0);
    float* sc = a.score + static_cast<size_t>(l) * a.plane + it.base + j;
    const float a_ld = *sc;
    const size_t cbase = (row0 + c) * Hq;
    const uint16_t* pp = part.p + cbase * CHUNK + tk;
    uint16_t pr[FOLD_HEADS];
#pragma unroll
    for (int q = 0; q < FOLD_HEADS; ++q) pr[q] = pp[min(q, Hq - 1) * CHUNK];
    const float m_own = part.ml[cbase + min(t % FOLD_HEADS, Hq - 1)].x;

    // the layer statistics of every head: row group rg of head h takes
    // chunks rg, rg + OUT_ROWS, ... with a running max, then the groups merge
#pragma unroll
    for (int u = 0; u < FINISH_PAIRS; ++u) {
        const int pi = t + u * OUT_THREADS;
        if (pi < Hq * OUT_ROWS) {
            const int rg = pi % OUT_ROWS;
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
            s_gm[pi] = M;
            s_gl[pi] = S;
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
    // grids of at most two workgroups per CU: four tiles in flight per wave
    // (all eight measured slower: their registers spill into the AGPRs)
    if (static_cast<int64_t>(a.L) * a.n_chunks <= ATTEND_DEEP_MAX_ITEMS)
        hipLaunchKernelGGL((decode_attend_kernel<NW, RAG, PAIRS>), dim3(a.L * a.n_chunks), dim3(64 * NW), 0, stream, a);
    else
        hipLaunchKernelGGL((decode_attend_kernel<NW, RAG, 1>), dim3(a.L * a.n_chunks), dim3(64 * NW), 0, stream, a);
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
