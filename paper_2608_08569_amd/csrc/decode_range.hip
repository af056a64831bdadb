// Decode step (Sec. 3.1 Eq. 1-2, Sec. 3.2.2 Eq. 6), whole-range path: for a
// call over many (layer, KV head) items, one workgroup per item streams every
// key of a sequence (or of an 8192-key part of a longer one), so no per-chunk
// partial results leave the chip.
// Compiled with the max-ILP machine scheduler (per-file flag of the build):
// the default one over-subscribes the 256 registers per lane and spills.
#include <atomic>

#include "decode_mfma.h"
#include "select.h"

namespace {

using namespace vz_mfma;

// ---- whole-range path: calls over many (layer, KV head) items ----
// One workgroup of RW waves per (layer, KV head) streams every key of the
// head (of a sequence, or of one part of it), so the softmax of its query
// heads completes inside the workgroup:
// wave w takes a contiguous run of about 1 / RW of the full 128-key chunks
// (contiguous runs stream about 7 % faster than chunks dealt round-robin to
// the waves), and wave 0 also the last, partial chunk: the first wave of each
// SIMD gets the memory pipe first and finishes tens of microseconds ahead of
// the second, so work added to it stays off the critical path.  Each wave
// keeps, per head, a running
// max, sum and output (online softmax, the output rescaled whenever the max
// grows), plus each chunk's p~ = exp2(s - m_ref) in bfloat16 (the
// first RLDS chunks in LDS, the others in registers) and the reference max
// m_ref it was taken against.  At the end
// the waves merge their (max, sum) pairs and outputs in LDS, the workgroup
// writes its query heads' output rows, and every key's sum over those heads
// of p_hj goes to the workspace.  For a sequence in one part, the last of a
// layer's workgroups to finish then adds the KV heads' sums into Eq. (6) and,
// in a generation step, runs the eviction of Sec. 3.2.2 for the layer (see
// arrive_last); no workgroup ever waits for another.  For ragged calls a fold
// kernel adds the sums.  A part of a longer sequence instead leaves its statistics,
// output and per-head probabilities relative to its own max, which a merge
// kernel and the fold combine.  Compared with the chunked path there are no
// per-chunk partial outputs or probabilities in HBM; it needs enough (layer,
// KV head) items to occupy the GPU, one workgroup per CU.
constexpr int RW = 8;                              // waves per workgroup (256 registers per lane)
constexpr int RFULL = 8;                           // full chunks per wave
constexpr int RNCH = RFULL + 1;                    // ... plus a last chunk of at most VT keys
constexpr int RLDS = 5;                            // chunks whose p~ waits in LDS (the rest in registers)
constexpr int RANGE_MAX_KEYS = RW * RFULL * CHUNK + VT;  // 8224 keys: T = B + 1 for budgets up to 8223
constexpr int RPART = RW * RFULL * CHUNK;          // 8192: longest part of a longer sequence
constexpr int RANGE_MIN_ITEMS = 128;               // (layer, KV head) items for the whole-range path
constexpr int RANGE_MAX_SEQS = 1024;               // sequences a ragged call ranks longest first (one order block)
constexpr int RO_STRIDE = D + 4;                   // padded LDS row of a wave's output (floats)
constexpr int RFOLD_KEYS = 256;                    // keys per fold block; parts are multiples of it

inline __host__ __device__ int64_t range_row(int64_t plane) { return (plane + CHUNK - 1) / CHUNK * CHUNK; }

// Parts of a sequence of T keys in a call of `items` (layer, KV head) items
// on `cus` compute units: one part when T <= RANGE_MAX_KEYS; else P0 =
// ceil(T / RPART) parts, or, when P0 >= 3, P0 + 1 if that makes
// ceil(items P / cus) * ceil(T / P) -- whole rounds of one workgroup per CU
// times the part length -- smaller, so that the last round of workgroups is
// not left to a fraction of the CUs (48 x 4 items at 24,576 keys: 4 parts,
// 3 full rounds, instead of 3 parts, 2.25 rounds; with 2 parts the model
// never prefers 3).  At most one part more, and only past 2 RPART keys,
// keeps a ragged call's work table small: its empty workgroups cost launch
// slots.  Then parts of kp keys (a multiple of RFOLD_KEYS,
// at most RPART), the last one holding the remaining T - (P - 1) kp >= 1
// keys.  A ragged call uses the same function, so a sequence is split the
// same way as in a single-sequence call of the same layers and KV heads.
__host__ __device__ inline void range_parts(int T, int items, int cus, int& P, int& kp) {
    if (T <= RANGE_MAX_KEYS) {
        P = 1;
        kp = T;
        return;
    }
    const int p0 = (T + RPART - 1) / RPART;
    int best = p0;
    if (p0 >= 3 && items > 0 && cus > 0) {
        long long best_cost = -1;
        for (int p = p0; p <= p0 + 1; ++p) {
            const long long rounds = (static_cast<long long>(items) * p + cus - 1) / cus;
            const long long cost = rounds * ((T + p - 1) / p);
            if (best_cost < 0 || cost < best_cost) {
                best_cost = cost;
                best = p;
            }
        }
    }
    kp = ((T + best - 1) / best + RFOLD_KEYS - 1) / RFOLD_KEYS * RFOLD_KEYS;
    P = (T + kp - 1) / kp;
}
// Fold blocks of such a sequence (one per RFOLD_KEYS keys of each part).
__host__ __device__ inline int range_fold_blocks(int T, int P, int kp) {
    if (P == 1) return (T + RFOLD_KEYS - 1) / RFOLD_KEYS;
    return (P - 1) * (kp / RFOLD_KEYS) + (T - (P - 1) * kp + RFOLD_KEYS - 1) / RFOLD_KEYS;
}

// One work item of the path: keys [k0, k1) of sequence s, part p of P.
struct RangeItem {
    int32_t s, p, P, kp;
    int32_t k0, k1, len, next_pos;
    int64_t base;  // first slot of the sequence in the planes
    int32_t pad[6];
};
static_assert(sizeof(RangeItem) == 64, "one 64-byte record per item");

// Workspace after the header (every array on a 256-byte boundary):
//   sums  [L][Hkv][row] float          per key, the sum over the KV head's query
//                                      heads of p_hj (sequences of one part;
//                                      rows padded to whole chunks)
//   rows  [L][Hkv][row][GMAX] bf16     per key and query head, p_hj relative to
//                                      its part's max (sequences of several parts)
//   pstat [L][Hkv][R][GMAX] float2     each part's max and sum of exp2, per head
//   pout  [L][Hkv][R][GMAX][D] float   each part's output relative to its max
//   ftab  [L][R][Hq] float             exp2(m_part - M) / S per part and head
//   items [R] RangeItem                a ragged call's parts, in dispatch order
//   fblk  [FB] int2                    a ragged call's fold blocks: (item, first key)
//   mlist [MB] int32                   a ragged call's sequences in several parts:
//                                      the item of each one's first part
// The parts' arrays exist when a sequence can have several parts (planes of
// more than RANGE_MAX_KEYS slots), the tables in ragged calls only.  A ragged
// call keeps its table sizes (items, fold blocks, sequences in parts) in the
// header.
struct RangeWs {
    float* sums;
    uint16_t* rows;
    float2* pstat;
    float* pout;
    float* ftab;
    RangeItem* items;
    int2* fblk;
    int32_t* mlist;
    int32_t* counts;  // [3] in the header: items, fold blocks, sequences in parts
    int64_t row;
};
__host__ __device__ inline size_t ws_align(size_t x) { return (x + 255) / 256 * 256; }
// Byte offsets of the arrays from the start of the workspace; returns the end.
__host__ __device__ inline size_t range_layout(size_t hdr, int L, int NW, int Hq, int64_t plane, int R, int FB,
                                               int MB, bool ragged, size_t off[8]) {
    const size_t row = static_cast<size_t>(range_row(plane));
    const size_t heads = static_cast<size_t>(L) * NW;
    const bool parts = plane > RANGE_MAX_KEYS;
    size_t o = ws_align(hdr);
    off[0] = o;
    o = ws_align(o + heads * row * sizeof(float));
    off[1] = o;
    if (parts) o = ws_align(o + heads * row * GMAX * sizeof(uint16_t));
    off[2] = o;
    if (parts) o = ws_align(o + heads * R * GMAX * sizeof(float2));
    off[3] = o;
    if (parts) o = ws_align(o + heads * R * GMAX * D * sizeof(float));
    off[4] = o;
    if (parts) o = ws_align(o + static_cast<size_t>(L) * R * Hq * sizeof(float));
    off[5] = o;
    if (ragged) o = ws_align(o + static_cast<size_t>(R) * sizeof(RangeItem));
    off[6] = o;
    if (ragged) o = ws_align(o + static_cast<size_t>(FB) * sizeof(int2));
    off[7] = o;
    if (ragged) o = ws_align(o + static_cast<size_t>(MB) * sizeof(int32_t));
    return o;
}
template <int NW>
__device__ __forceinline__ RangeWs range_ws(const FusedArgs& a, bool ragged) {
    size_t off[8];
    range_layout(a.hdr_bytes, a.L, NW, a.Hq, a.plane, a.R, a.FB, a.MB, ragged, off);
    RangeWs w;
    w.sums = reinterpret_cast<float*>(a.ws + off[0]);
    w.rows = reinterpret_cast<uint16_t*>(a.ws + off[1]);
    w.pstat = reinterpret_cast<float2*>(a.ws + off[2]);
    w.pout = reinterpret_cast<float*>(a.ws + off[3]);
    w.ftab = reinterpret_cast<float*>(a.ws + off[4]);
    w.items = reinterpret_cast<RangeItem*>(a.ws + off[5]);
    w.fblk = reinterpret_cast<int2*>(a.ws + off[6]);
    w.mlist = reinterpret_cast<int32_t*>(a.ws + off[7]);
    w.counts = reinterpret_cast<int32_t*>(a.ws);
    w.row = range_row(a.plane);
    return w;
}

// Item r of a single-sequence call (parts of a.part_keys keys).
__device__ __forceinline__ RangeItem single_item(const FusedArgs& a, int r) {
    RangeItem it;
    it.s = 0;
    it.p = r;
    it.P = a.n_parts;
    it.kp = a.part_keys;
    it.k0 = r * a.part_keys;
    it.k1 = min(a.len + 1, it.k0 + a.part_keys);
    it.len = a.len;
    it.next_pos = a.next_pos;
    it.base = 0;
    return it;
}

// Row of key r (0..CHUNK-1) in a chunk's [key][head] bfloat16 rows
// (16 bytes each): bit 1 is flipped by bit 4, so that the 8 keys one write
// instruction covers (r = c + 4 q4 + 16 hi) start on 8 distinct 4-bank groups.
__device__ __forceinline__ int pslot(int r) { return r ^ ((r >> 3) & 2); }

// Wave-uniform copy of an item (its fields feed scalar buffer descriptors).
__device__ __forceinline__ RangeItem uniform_item(const RangeItem& x) {
    RangeItem it;
    it.s = __builtin_amdgcn_readfirstlane(x.s);
    it.p = __builtin_amdgcn_readfirstlane(x.p);
    it.P = __builtin_amdgcn_readfirstlane(x.P);
    it.kp = __builtin_amdgcn_readfirstlane(x.kp);
    it.k0 = __builtin_amdgcn_readfirstlane(x.k0);
    it.k1 = __builtin_amdgcn_readfirstlane(x.k1);
    it.len = __builtin_amdgcn_readfirstlane(x.len);
    it.next_pos = __builtin_amdgcn_readfirstlane(x.next_pos);
    const uint64_t b = static_cast<uint64_t>(x.base);
    it.base = static_cast<int64_t>(
        static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b)))) |
        (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b >> 32)))) << 32));
    return it;
}

// Arrival of one workgroup of a layer (thread 0, after every store the others
// need has completed): a lock-free compare-and-swap on the layer's counter,
// whose high word is the call's tag and whose low word counts this call's
// arrivals.  A counter holding another tag (an earlier call, or memory never
// used) counts as zero, so the workspace needs no initialisation.  Returns
// true for the n-th arrival, which also resets the counter to 0 (a graph
// replaying the call with the same tag starts from zero again).  Relaxed
// device-scope atomics: the data the last arriver reads was written with
// device-coherent stores that completed before the arrivals.
__device__ __forceinline__ bool arrive_last(uint64_t* c, uint32_t tag, uint32_t n) {
    uint64_t cur = __hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    uint64_t want;
    do {
        want = (static_cast<uint32_t>(cur >> 32) == tag ? cur : static_cast<uint64_t>(tag) << 32) + 1;
    } while (!__hip_atomic_compare_exchange_weak(c, &cur, want, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT));
    const bool last = static_cast<uint32_t>(want) == n;
    if (last) __hip_atomic_store(c, uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return last;
}

// Grid (NW, L) for a sequence of one part; NW x L x items, flattened, for
// parts and ragged calls (KV head fastest, then layer, then item, so a
// ragged call's items go out in the table's order): workgroup (g, l, r)
// takes KV head g of layer l over the keys of item r.  RAG: items from the
// ragged call's table (dispatch order longest first); else the parts of the
// single sequence.  SPLIT: items may be parts of a longer sequence, whose
// statistics, outputs and per-head probabilities go to the workspace for the
// merge and fold kernels.  Neither (a single sequence in one part): the
// layer's last workgroup folds the scores and evicts (fold_select_layer).
template <int NW, bool RAG, bool SPLIT>
__global__ __launch_bounds__(64 * RW, 1) void decode_range_kernel(const FusedArgs a) {
    constexpr bool FS = !RAG && !SPLIT;
    static_assert(RW * GMAX * RO_STRIDE * 4 <= RW * TILE_BYTES, "the merged outputs fit in the tile buffers");
    __shared__ __attribute__((aligned(16))) uint8_t s_tile[RW][TILE_BYTES];
    __shared__ float2 s_stat[RW][GMAX];
    // p~ of the first RLDS chunks of each wave, transposed: [slot(key)][head]
    // in bfloat16 (16 bytes per key; slot() in the head-sum epilogue)
    __shared__ __attribute__((aligned(16))) uint16_t s_pt[RW][RLDS][CHUNK][GMAX];
    __shared__ __attribute__((aligned(16))) float s_mref[RW][RNCH][GMAX];  // reference max of each chunk's p~, per head (then its factor)
    __shared__ float2 s_MS[GMAX];             // the workgroup's max M and 1 / sum S, per head
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int q4 = lane >> 4, r16 = lane & 15;
    const int hi = r16 >> 3, hh = r16 & 7;
    const int Hq = a.Hq, G = Hq / NW;
    constexpr bool FLAT = RAG || SPLIT;
    const int g = FLAT ? static_cast<int>(blockIdx.x) % NW : static_cast<int>(blockIdx.x);
    const int l = FLAT ? (static_cast<int>(blockIdx.x) / NW) % a.L : static_cast<int>(blockIdx.y);
    // (a single sequence in parts takes them last to first on odd steps, as
    // the waves their chunks below: the parts a step reads last, in its last
    // round of workgroups, are then the first the next step reads)
    const int r0 = FLAT ? static_cast<int>(blockIdx.x) / (NW * a.L) : 0;
    const int r = !RAG && SPLIT && (a.next_pos & 1) ? a.n_parts - 1 - r0 : r0;
    const RangeWs rws = range_ws<NW>(a, RAG);
    RangeItem it;
    if constexpr (RAG) {
        if (r >= rws.counts[0]) return;
        it = uniform_item(rws.items[r]);
    } else {
        it = single_item(a, r);
    }
    const bool split = SPLIT && it.P > 1;
    const int len = it.len;
    const int NK = it.k1 - it.k0;             // keys of this item
    const int n_full = NK / CHUNK;            // full chunks; chunk n_full holds the other NK % CHUNK keys
    const bool part = NK % CHUNK != 0;
    // Steps whose new position is odd read the chunks in the other
    // direction (see chunk_of below) and, where wave 0's last slot allows it,
    // with the two halves of the waves' ranges exchanged: the first wave of
    // each SIMD, which gets the memory pipe first, then starts on the range
    // the second one read last in the previous step.
    const bool odd = (it.next_pos & 1) != 0;
    const int half = RW / 2;
    const int s_half = ((half + 1) * n_full) / RW - (half * n_full) / RW;  // full chunks of range RW / 2
    const bool swap = odd && (s_half < RFULL || NK % CHUNK <= VT);  // wave 0 keeps the partial chunk
    const int wr = swap ? (w ^ half) : w;  // the wave's range
    const int c0 = __builtin_amdgcn_readfirstlane(wr * n_full / RW);  // the wave's full chunks: [c0, c0 + my_full)
    const int my_full = __builtin_amdgcn_readfirstlane((wr + 1) * n_full / RW - c0);
    const int my_chunks = my_full + (w == 0 && part ? 1 : 0);
    // Chunk of the wave's slot k.  Range 0 has the fewest full chunks
    // (n_full / RW), so on wave 0 the partial chunk is at most its slot
    // RFULL, and there only when n_full = RW * RFULL, where the part limit
    // (RANGE_MAX_KEYS keys for a whole sequence, RPART for a part of a longer
    // one) leaves it <= VT keys; with the ranges exchanged, wave 0 holds range
    // RW / 2, which the condition on `swap` keeps to the same bound.
    // Odd steps take the full chunks of every wave in reverse order:
    // consecutive steps of a sequence re-read the same cache, and the keys a
    // step reads last are then the first the next step reads, while they are
    // still in the memory-side cache (Infinity Cache).  The order follows from
    // the call's arguments, so a step's bits do too.
    auto chunk_of = [&](int k) { return k < my_full ? (odd ? c0 + my_full - 1 - k : c0 + k) : n_full; };
    const size_t seq_row = static_cast<size_t>(it.s) * a.L + l;  // (sequence, layer) row of q, out, k_new, v_new
    const size_t head_base = ((static_cast<size_t>(l) * NW + g) * a.plane + it.base + it.k0) * D;
    uint16_t* Kh = a.k_cache + head_base;  // the item's first key
    uint16_t* Vh = a.v_cache + head_base;

    // Eq. (1) first: in the last part, the wave whose chunks hold slot len
    // (the partial chunk's wave 0, else the wave holding range RW - 1) writes
    // the new row before any of its loads, so every key is read from the
    // cache alike.
    if (it.p == it.P - 1 && w == (part ? 0 : (RW - 1) ^ (swap ? half : 0))) {
        const uint16_t* kn = a.k_new + (seq_row * NW + g) * D;
        const uint16_t* vn = a.v_new + (seq_row * NW + g) * D;
        const size_t at = static_cast<size_t>(len - it.k0) * D;
        if (lane < 16)
            *reinterpret_cast<uint4*>(Kh + at + 8 * lane) = *reinterpret_cast<const uint4*>(kn + 8 * lane);
        else if (lane < 32)
            *reinterpret_cast<uint4*>(Vh + at + 8 * (lane - 16)) = *reinterpret_cast<const uint4*>(vn + 8 * (lane - 16));
        // (with FS the last workgroup of the layer writes the position)
        if (!FS && g == 0 && lane == 0) a.pos[static_cast<size_t>(l) * a.plane + it.base + len] = it.next_pos;
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
        const int nk = live ? min(CHUNK, NK - c * CHUNK) : 0;
        const int u = j & 3;
        const int rows = nk - VT * u > 0 ? nk - VT * u : 0;
        const uint16_t* base = (j < 4 ? Kh : Vh) + (static_cast<size_t>(c) * CHUNK + VT * u) * D;
        // (the byte bound through readfirstlane: in a vector register it would
        // make the compiler wrap each load in a loop over the lanes' descriptors)
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t*>(base), 0, __builtin_amdgcn_readfirstlane(rows * D * 2), kBufferDword3);
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
        const uint16_t* qrow = a.q + (seq_row * Hq + g * G + hq) * D + 8 * q4;
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
    // p~ of chunks RLDS.. RFULL - 1 in registers (bfloat16 pairs); a wave's
    // chunk RFULL exists only as the last chunk of a cache with more than
    // RW * RFULL full chunks, which has at most VT keys: one 32-key tile.
    uint32_t pst[RFULL - RLDS][2 * PAIRS];
    uint32_t pst_last[2];

#pragma unroll
    for (int k = 0; k < RNCH; ++k) {
        if (k < my_chunks) {
        const int c = chunk_of(k);
        const int nk = min(CHUNK, NK - c * CHUNK);
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
            pk[2 * u] = pack_bf16x2(sp[u][0], sp[u][1]);
            pk[2 * u + 1] = pack_bf16x2(sp[u][2], sp[u][3]);
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

    // The layer's old scores and positions for the fold of its last
    // workgroup, in flight during the epilogue (loads are counted in order
    // with the stores, so issued here they are back before the arrival waits
    // for the head-group sums' stores).
    constexpr int FB = (RANGE_MAX_KEYS + 64 * RW - 1) / (64 * RW);        // slots per thread
    constexpr int FR = (RANGE_MAX_KEYS + 4 * 64 * RW - 1) / (4 * 64 * RW);  // rounds of 4 slots per thread
    vz_sel::FoldOld<FB> old;
    if constexpr (FS)
        vz_sel::fold_prefetch<64 * RW, FB>(a.score + static_cast<size_t>(l) * a.plane,
                                            a.pos + static_cast<size_t>(l) * a.plane, len + 1, old);

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
    // a part of a longer sequence keeps its output and p~ relative to its own
    // max; the merge kernel applies the sequence's statistics
    const float inv_S = split ? 1.f : 1.0f / S;
    if (w == 0 && q4 == 0 && hi == 0) s_MS[hh] = make_float2(M, inv_S);  // read after the next barrier
    const size_t part_row = (static_cast<size_t>(l) * NW + g) * a.R + r;  // (layer, KV head, item) of pstat, pout
    if (split && w == 0 && q4 == 0 && hi == 0 && hh < G) rws.pstat[part_row * GMAX + hh] = make_float2(M, S);

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
        if (split)
            rws.pout[(part_row * GMAX + h) * D + ch] = o;
        else
            a.out[(seq_row * Hq + g * G + h) * D + ch] = vz::f32_to_bf16(o);
    }

    // ---- each key's sum over this KV head's query heads of p_hj ----
    // Every chunk's p~ ends up as [slot(key)][head] bfloat16 rows: the
    // LDS-resident chunks were written so in the loop, the register-held ones
    // are written to the wave's (now free) tile buffer here.  Each lane then
    // reads two keys' rows and forms sum_h p~_h * f_h with f_h =
    // exp2(m_ref,h - M_h) / S_h from a per-chunk factor table.  (LDS
    // operations of a wave complete in order: no barrier between a wave's own
    // writes and reads.)
    __syncthreads();  // the output merge has read the tile buffers; s_MS is written
    const size_t key0 = (static_cast<size_t>(l) * NW + g) * rws.row + it.base + it.k0;  // the item's first key
    float* const gsum = rws.sums + key0;
    uint16_t* const prow = rws.rows + key0 * GMAX;
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
            for (int x = 0; x < RFULL - RLDS; ++x)  // register slots: fixed indexes, wave-uniform choice
                if (k == RLDS + x) {
#pragma unroll
                    for (int i = 0; i < 2 * PAIRS; ++i) pk[i] = pst[x][i];
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
        const int kk = chunk_of(k) * CHUNK + 2 * lane;  // the lane's first key in the item
        if (split) {
            // each key's row of p~ f_h (relative to the part's max), bfloat16
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const uint4 rw = *reinterpret_cast<const uint4*>(rows + pslot(2 * lane + e) * GMAX);
                const uint32_t wd[4] = {rw.x, rw.y, rw.z, rw.w};
                uint32_t ow[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) ow[i] = pack_bf16x2(bf16_lo(wd[i]) * fk[2 * i], bf16_hi(wd[i]) * fk[2 * i + 1]);
                if (kk + e < NK)
                    *reinterpret_cast<uint4*>(prow + static_cast<size_t>(kk + e) * GMAX) = make_uint4(ow[0], ow[1], ow[2], ow[3]);
            }
        } else {
            float y[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const uint4 rw = *reinterpret_cast<const uint4*>(rows + pslot(2 * lane + e) * GMAX);
                const uint32_t wd[4] = {rw.x, rw.y, rw.z, rw.w};
                float acc = 0.f;
#pragma unroll
                for (int h = 0; h < GMAX; ++h) acc = fmaf((h & 1) ? bf16_hi(wd[h >> 1]) : bf16_lo(wd[h >> 1]), fk[h], acc);
                y[e] = acc;
            }
            if constexpr (RAG) {
                // slots past the item belong to the next sequence: masked
                if (kk < NK) gsum[kk] = y[0];
                if (kk + 1 < NK) gsum[kk + 1] = y[1];
            } else if constexpr (FS) {
                // device-coherent: another workgroup of this kernel folds them
                const uint64_t pair = static_cast<uint64_t>(__float_as_uint(y[0])) |
                                      (static_cast<uint64_t>(__float_as_uint(y[1])) << 32);
                __hip_atomic_store(reinterpret_cast<uint64_t*>(gsum + kk), pair, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            } else {
                *reinterpret_cast<float2*>(gsum + kk) = make_float2(y[0], y[1]);
            }
        }
    }
    if constexpr (FS) {
        // ---- the layer's last workgroup: Eq. (6) fold, then the eviction ----
        using Sel = vz_sel::SelShared<64 * RW, FB * 64 * RW>;
        static_assert(sizeof(Sel) <= sizeof(s_pt), "the selection's LDS fits in the p~ rows");
        static_assert((4 * FR + 2) * 64 * RW * 4 <= sizeof(s_tile) && FB <= 4 * FR, "the summed sums fit in the tiles");
        __shared__ int s_last;
        vz_sel::FoldLayer<uint16_t> f;
        const size_t lrow = static_cast<size_t>(l) * a.plane;
        f.A = a.score + lrow;
        f.P = a.pos + lrow;
        f.k0 = a.k_cache + lrow * NW * D;
        f.v0 = a.v_cache + lrow * NW * D;
        f.head_stride = static_cast<size_t>(a.plane) * D;
        f.S = rws.sums + static_cast<size_t>(l) * NW * rws.row;
        f.row = rws.row;
        f.k_new = a.k_new + seq_row * NW * D;
        f.v_new = a.v_new + seq_row * NW * D;
        f.len = len + 1;
        f.next_pos = it.next_pos + 1;
        f.gamma = a.gamma;
        f.select = a.ev != 0;
        f.budget = a.ev_budget;
        f.n_sink = a.ev_sink;
        f.M = a.ev_M;
        f.kept = a.ev_kept ? a.ev_kept + static_cast<size_t>(l) * a.ev_budget : nullptr;
        f.n_out = a.ev_n ? a.ev_n + l : nullptr;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's sums have reached the device
        __syncthreads();
        if (tid == 0) s_last = arrive_last(a.cnt + l, a.tag, NW);
        __syncthreads();
        if (!s_last) return;
        Sel& sh = *reinterpret_cast<Sel*>(&s_pt[0][0][0][0]);             // the p~ rows are no longer read
        float* const s_acc = reinterpret_cast<float*>(&s_tile[0][0]);      // nor the tiles
        vz_sel::fold_select_layer<64 * RW, FB, FR, VZ_BF16, D, NW>(f, old, s_acc, sh);
    }
}

// Merge of a sequence in parts, one block per (sequence in parts, layer,
// pair of query heads) -- a ragged call's sequences in parts are listed by
// the order kernel, a single sequence is item 0 -- and thread t takes
// channel t % D of head 2 hb + t / D.  Per head, the sequence's max M and sum S from the parts'
// pairs, each part's factor exp2(m_part - M) / S (kept for the fold), and the
// output row, the parts' outputs times their factors, added in part order.
// (Every thread of a head forms M, S and the factors itself, from the same
// few pairs; a block per (sequence, layer) over all heads left the call's
// merge on 48 CUs at a time.)
constexpr int RMERGE_THREADS = 2 * D;
constexpr int RMERGE_HEADS = RMERGE_THREADS / D;
template <int NW, bool RAG>
__global__ __launch_bounds__(RMERGE_THREADS) void range_merge_kernel(const FusedArgs a) {
    const int l = blockIdx.y, t = threadIdx.x;
    const RangeWs rws = range_ws<NW>(a, RAG);
    int r = 0;
    RangeItem it;
    if constexpr (RAG) {
        if (static_cast<int>(blockIdx.x) >= rws.counts[2]) return;
        r = rws.mlist[blockIdx.x];
        it = rws.items[r];
    } else {
        it = single_item(a, r);
    }
    if (it.P == 1 || it.p != 0) return;
    const int Hq = a.Hq, G = Hq / NW, P = it.P;
    const int h = static_cast<int>(blockIdx.z) * RMERGE_HEADS + t / D, ch = t % D;
    if (h >= Hq) return;
    const int g = h / G, hg = h - g * G;
    const float2* ps = rws.pstat + ((static_cast<size_t>(l) * NW + g) * a.R + r) * GMAX + hg;
    float M = -INFINITY;
    for (int p = 0; p < P; ++p) M = fmaxf(M, ps[static_cast<size_t>(p) * GMAX].x);
    float S = 0.f;
    for (int p = 0; p < P; ++p) {
        const float2 x = ps[static_cast<size_t>(p) * GMAX];
        S = fmaf(x.y, exp2f(x.x - M), S);
    }
    const float inv_S = 1.0f / S;
    const float* po = rws.pout + (((static_cast<size_t>(l) * NW + g) * a.R + r) * GMAX + hg) * D + ch;
    float o = 0.f;
    for (int p = 0; p < P; ++p) {
        const float f = exp2f(ps[static_cast<size_t>(p) * GMAX].x - M) * inv_S;
        if (ch == 0) rws.ftab[(static_cast<size_t>(l) * a.R + r + p) * Hq + h] = f;
        o = fmaf(po[static_cast<size_t>(p) * GMAX * D], f, o);
    }
    a.out[((static_cast<size_t>(it.s) * a.L + l) * Hq + h) * D + ch] = vz::f32_to_bf16(o);
}

// Fold kernel of a ragged call or of a sequence in parts, one block of
// RFOLD_KEYS threads per fold block (keys of one item), thread = key: Eq. (6)
// from the KV heads' sums added in head order (a sequence of one part, the
// same arithmetic as the single-part fold kernel), or from each key's
// per-head rows and its part's factors.
template <int NW, bool RAG>
__global__ __launch_bounds__(RFOLD_KEYS) void range_fold_parts_kernel(const FusedArgs a) {
    __shared__ float s_f[NW * GMAX];
    const int b = blockIdx.x, l = blockIdx.y, t = threadIdx.x;
    const RangeWs rws = range_ws<NW>(a, RAG);
    int r, j0;
    RangeItem it;
    if constexpr (RAG) {
        if (b >= rws.counts[1]) return;
        const int2 e = rws.fblk[b];
        r = e.x;
        j0 = e.y;
        it = rws.items[r];
    } else {
        const int bpp = a.part_keys / RFOLD_KEYS;
        r = min(b / bpp, a.n_parts - 1);
        j0 = r * a.part_keys + (b - r * bpp) * RFOLD_KEYS;
        it = single_item(a, r);
        if (j0 >= it.k1) return;
    }
    const int len = it.len;
    const int jj = j0 + t;
    const int j = min(jj, it.k1 - 1);  // clamped: every load in bounds, the store masked
    const size_t slot = static_cast<size_t>(it.base) + j;
    float* const sc = a.score + static_cast<size_t>(l) * a.plane + slot;
    const float a_ld = *sc;
    float acc;
    if (it.P == 1) {
        const float* gs = rws.sums + static_cast<size_t>(l) * NW * rws.row + slot;
        acc = gs[0];
#pragma unroll
        for (int g = 1; g < NW; ++g) acc += gs[g * rws.row];
    } else {
        const int Hq = a.Hq, G = Hq / NW;
        uint4 rw[NW];
#pragma unroll
        for (int g = 0; g < NW; ++g)
            rw[g] = *reinterpret_cast<const uint4*>(rws.rows + ((static_cast<size_t>(l) * NW + g) * rws.row + slot) * GMAX);
        if (t < NW * GMAX) {
            const int g = t / GMAX, hg = t - g * GMAX;
            s_f[t] = hg < G ? rws.ftab[(static_cast<size_t>(l) * a.R + r) * Hq + g * G + hg] : 0.f;
        }
        __syncthreads();
        acc = 0.f;
#pragma unroll
        for (int g = 0; g < NW; ++g) {
            const uint32_t wd[4] = {rw[g].x, rw[g].y, rw[g].z, rw[g].w};
#pragma unroll
            for (int h = 0; h < GMAX; ++h)
                acc = fmaf((h & 1) ? bf16_hi(wd[h >> 1]) : bf16_lo(wd[h >> 1]), s_f[g * GMAX + h], acc);
        }
    }
    const float a_old = j < len ? a_ld : 0.f;  // zero pad of Eq. (6) for the new slot
    if (jj < it.k1) *sc = fmaf(a.gamma, a_old, acc);
}

// Work order of a ragged call, one block: every served sequence's parts,
// those of the longest parts first (ties: the smaller sequence index), so
// that the workgroups starting last are the short ones; the fold blocks of
// each part; each sequence's status.  A sequence that cannot be served, or
// whose parts would not fit the tables (sequences overlapping in the planes),
// is skipped and its status says why.  Batches of more than ORDER_THREADS
// sequences keep the sequence order instead (each thread a run of
// sequences, a block scan for the first item and fold block of each run).
constexpr int ORDER_THREADS = RANGE_MAX_SEQS;

// Parts and fold blocks of sequence s (0 when it cannot be served).
template <int NW>
__device__ __forceinline__ void order_seq(const FusedArgs& a, int s, int& st, int& T, int& P, int& kp, int& F) {
    T = P = kp = F = 0;
    st = vz::ragged_decode_status(a.rag, s);
    if (st == VZ_OK) {
        T = a.rag.len[s] + 1;
        range_parts(T, a.L * NW, a.cus, P, kp);
        F = range_fold_blocks(T, P, kp);
    }
}

// Items r0 .. r0 + P - 1 and fold blocks fb0 .. fb0 + F - 1 of sequence s.
__device__ void order_write(const FusedArgs& a, const RangeWs& rws, int s, int T, int P, int kp, int r0, int fb0,
                            bool fold_entries) {
    RangeItem it{};
    it.s = s;
    it.P = P;
    it.kp = kp;
    it.len = T - 1;
    it.next_pos = a.rag.next_pos[s];
    it.base = a.rag.base[s];
    int fb = fb0;
    for (int p = 0; p < P; ++p) {
        it.p = p;
        it.k0 = p * kp;
        it.k1 = min(T, (p + 1) * kp);
        rws.items[r0 + p] = it;
        if (fold_entries)
            for (int j0 = it.k0; j0 < it.k1; j0 += RFOLD_KEYS) rws.fblk[fb++] = make_int2(r0 + p, j0);
    }
}

template <int NW>
__device__ void order_in_sequence_order(const FusedArgs& a, const RangeWs& rws, int* s_a, int* s_b, int* s_c,
                                        int* s_n) {
    const int n = a.rag.n, t = threadIdx.x;
    const int per = (n + ORDER_THREADS - 1) / ORDER_THREADS;
    const int s0 = min(t * per, n), s1 = min(s0 + per, n);
    int sumP = 0, sumF = 0, sumM = 0;
    for (int s = s0; s < s1; ++s) {
        int st, T, P, kp, F;
        order_seq<NW>(a, s, st, T, P, kp, F);
        sumP += P;
        sumF += F;
        sumM += P > 1;
    }
    // exclusive block scan of the runs' items, fold blocks and sequences in parts
    s_a[t] = sumP;
    s_b[t] = sumF;
    s_c[t] = sumM;
    __syncthreads();
    for (int o = 1; o < ORDER_THREADS; o <<= 1) {
        const int xa = t >= o ? s_a[t - o] : 0, xb = t >= o ? s_b[t - o] : 0, xc = t >= o ? s_c[t - o] : 0;
        __syncthreads();
        s_a[t] += xa;
        s_b[t] += xb;
        s_c[t] += xc;
        __syncthreads();
    }
    int r = s_a[t] - sumP, fb = s_b[t] - sumF, m = s_c[t] - sumM;
    for (int s = s0; s < s1; ++s) {
        int st, T, P, kp, F;
        order_seq<NW>(a, s, st, T, P, kp, F);
        const bool fits = P > 0 && r + P <= a.R && fb + F <= a.FB && m + (P > 1) <= a.MB;
        if (P > 0 && !fits) st = VZ_ERR_CAPACITY;
        if (a.rag.status) a.rag.status[s] = st;
        if (fits) {
            order_write(a, rws, s, T, P, kp, r, fb, true);
            if (P > 1) rws.mlist[m] = r;
            atomicMax(&s_n[1], r + P);
            atomicMax(&s_n[2], fb + F);
            atomicMax(&s_n[3], m + (P > 1));
        }
        r += P;
        fb += F;
        m += P > 1;
    }
}

template <int NW>
__global__ __launch_bounds__(ORDER_THREADS) void range_order_kernel(const FusedArgs a) {
    __shared__ int s_kp[ORDER_THREADS], s_P[ORDER_THREADS], s_F[ORDER_THREADS];
    __shared__ int s_seq[ORDER_THREADS], s_fb[ORDER_THREADS], s_r0[ORDER_THREADS];
    __shared__ int s_n[4];  // sequences served, items, fold blocks, sequences in parts
    const RangeWs rws = range_ws<NW>(a, true);
    const int n = a.rag.n, t = threadIdx.x;
    if (t < 4) s_n[t] = 0;
    if (n > ORDER_THREADS) {
        __syncthreads();
        order_in_sequence_order<NW>(a, rws, s_kp, s_P, s_F, s_n);
        __syncthreads();
        if (t == 0) {
            rws.counts[0] = s_n[1];
            rws.counts[1] = s_n[2];
            rws.counts[2] = s_n[3];
        }
        return;
    }
    int st = VZ_OK, T = 0, P = 0, kp = 0, F = 0;
    if (t < n) {
        order_seq<NW>(a, t, st, T, P, kp, F);
        s_kp[t] = kp;
        s_P[t] = P;
        s_F[t] = F;
    }
    __syncthreads();
    // position among the served sequences, first item, first fold block,
    // sequences in parts before it
    int q = 0, r0 = 0, fb0 = 0, m0 = 0;
    if (P > 0) {
        for (int u = 0; u < n; ++u) {
            const int ku = s_kp[u];
            if (ku > kp || (ku == kp && u < t)) {
                ++q;
                r0 += s_P[u];
                fb0 += s_F[u];
                m0 += s_P[u] > 1;
            }
        }
    }
    // a sequence that does not fit pushes every later one out as well, so the
    // served ones hold positions 0 .. served - 1
    const bool fits = P > 0 && r0 + P <= a.R && fb0 + F <= a.FB && m0 + (P > 1) <= a.MB;
    if (P > 0 && !fits) st = VZ_ERR_CAPACITY;
    if (t < n && a.rag.status) a.rag.status[t] = st;
    if (fits) {
        s_seq[q] = t;
        s_fb[q] = fb0;
        s_r0[q] = r0;
        atomicAdd(&s_n[0], 1);
        atomicMax(&s_n[1], r0 + P);
        atomicMax(&s_n[2], fb0 + F);
        atomicMax(&s_n[3], m0 + (P > 1));
        if (P > 1) rws.mlist[m0] = r0;
        order_write(a, rws, t, T, P, kp, r0, fb0, false);  // fold entries below, spread over the block
    }
    __syncthreads();
    const int served = s_n[0], n_fold = s_n[2];
    for (int b = t; b < n_fold; b += ORDER_THREADS) {
        int lo = 0, hi = served - 1;  // the last position whose first fold block is <= b
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_fb[mid] <= b) lo = mid;
            else hi = mid - 1;
        }
        const int u = s_seq[lo], o = b - s_fb[lo];
        const int Pu = s_P[u], kpu = s_kp[u];
        const int bpp = Pu == 1 ? 1 : kpu / RFOLD_KEYS;
        const int p = Pu == 1 ? 0 : min(o / bpp, Pu - 1);
        rws.fblk[b] = make_int2(s_r0[lo] + p, p * kpu + (o - p * bpp) * RFOLD_KEYS);
    }
    if (t == 0) {
        rws.counts[0] = s_n[1];
        rws.counts[1] = n_fold;
        rws.counts[2] = s_n[3];
    }
}

// Item and fold-block bounds of a ragged call over `total` slots: a sequence
// of T keys has at most ceil(T / RPART) parts, one more past 2 RPART keys,
// and T / RFOLD_KEYS + (parts) fold blocks; the sequences' keys add up to at
// most `total`, so at most total / (2 RPART + 1) of them are that long.
int32_t ragged_items_bound(int32_t n_seqs, int64_t total) {
    const int64_t longs = total / (2 * RPART + 1);
    return static_cast<int32_t>(n_seqs + (total + RPART - 1) / RPART + (longs < n_seqs ? longs : n_seqs));
}
// Parts a single-sequence workspace holds for planes of `plane` slots.
int32_t single_parts_bound(int64_t plane) {
    const int64_t p0 = (plane + RPART - 1) / RPART;
    return static_cast<int32_t>(p0 >= 3 ? p0 + 1 : p0);
}
// Compute units of the current device (queried once per device).
int32_t device_cus() {
    static std::atomic<int32_t> cus[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int32_t n = cus[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        n = v;
        cus[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}
// Sequences of a ragged call that can be in several parts: more than
// RANGE_MAX_KEYS keys each, in non-overlapping slots of `total`.
int32_t ragged_multi_bound(int32_t n_seqs, int64_t total) {
    const int64_t longs = total / (RANGE_MAX_KEYS + 1);
    return static_cast<int32_t>(longs < n_seqs ? longs : n_seqs);
}
int32_t ragged_fold_bound(int32_t n_seqs, int64_t total) {
    return static_cast<int32_t>((total + RFOLD_KEYS - 1) / RFOLD_KEYS + ragged_items_bound(n_seqs, total));
}

template <int NW>
hipError_t launch_range(const FusedArgs& a, hipStream_t stream) {
    if (a.rag.n > 0) {
        hipLaunchKernelGGL((range_order_kernel<NW>), dim3(1), dim3(ORDER_THREADS), 0, stream, a);
        hipLaunchKernelGGL((decode_range_kernel<NW, true, true>), dim3(NW * a.L * a.R), dim3(64 * RW), 0, stream, a);
        if (a.MB > 0)
            hipLaunchKernelGGL((range_merge_kernel<NW, true>),
                               dim3(a.MB, a.L, (a.Hq + RMERGE_HEADS - 1) / RMERGE_HEADS), dim3(RMERGE_THREADS), 0,
                               stream, a);
        hipLaunchKernelGGL((range_fold_parts_kernel<NW, true>), dim3(a.FB, a.L), dim3(RFOLD_KEYS), 0, stream, a);
        return hipGetLastError();
    }
    if (a.n_parts > 1) {
        hipLaunchKernelGGL((decode_range_kernel<NW, false, true>), dim3(NW * a.L * a.n_parts), dim3(64 * RW), 0,
                           stream, a);
        hipLaunchKernelGGL((range_merge_kernel<NW, false>), dim3(1, a.L, (a.Hq + RMERGE_HEADS - 1) / RMERGE_HEADS),
                           dim3(RMERGE_THREADS), 0, stream, a);
        hipLaunchKernelGGL((range_fold_parts_kernel<NW, false>),
                           dim3(range_fold_blocks(a.len + 1, a.n_parts, a.part_keys), a.L), dim3(RFOLD_KEYS), 0,
                           stream, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((decode_range_kernel<NW, false, false>), dim3(NW, a.L), dim3(64 * RW), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

bool vz_decode_range_ok(int32_t L, int32_t Hkv, int32_t n_seqs) {
    (void)n_seqs;  // any batch: the order kernel ranks up to RANGE_MAX_SEQS sequences, keeps the order beyond
    return static_cast<int64_t>(L) * Hkv >= RANGE_MIN_ITEMS;
}

hipError_t vz_launch_decode_range(const FusedArgs& a0, int32_t Hkv, hipStream_t stream) {
    FusedArgs a = a0;
    a.cus = device_cus();
    if (a.rag.n > 0) {
        a.R = ragged_items_bound(a.rag.n, a.plane);
        a.FB = ragged_fold_bound(a.rag.n, a.plane);
        a.MB = ragged_multi_bound(a.rag.n, a.plane);
    } else {
        range_parts(a.len + 1, a.L * Hkv, a.cus, a.n_parts, a.part_keys);
        a.R = a.n_parts;
        a.FB = 0;
    }
    switch (Hkv) {
        case 1: return launch_range<1>(a, stream);
        case 2: return launch_range<2>(a, stream);
        case 4: return launch_range<4>(a, stream);
        case 8: return launch_range<8>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

bool vz_decode_range_whole(int32_t len) { return static_cast<int64_t>(len) + 1 <= RANGE_MAX_KEYS; }

size_t vz_decode_range_ws_bytes(int32_t L, int32_t Hq, int32_t Hkv, int64_t plane, int32_t n_seqs) {
    size_t off[8];
    const bool rag = n_seqs > 0;
    const int R = rag ? ragged_items_bound(n_seqs, plane) : single_parts_bound(plane);
    const int FB = rag ? ragged_fold_bound(n_seqs, plane) : 0;
    const int MB = rag ? ragged_multi_bound(n_seqs, plane) : 0;
    return range_layout(vz_decode_hdr_bytes(L), L, Hkv, Hq, plane, R, FB, MB, rag, off);
}

