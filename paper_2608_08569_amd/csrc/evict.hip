// Stage-2 eviction (Sec. 3.2.2, Eq. 7-9) with in-place hole-fill compaction.
//
// select kernel (one 1024-thread block per layer):
//   1. Rank key per slot: (order-preserving score bits << 32) | ~pos, so the
//      larger key is the more important slot (ties to the smaller position).
//      Only middle slots (not sink, not recent) compete.  E = len - budget of
//      them are evicted: the E smallest keys.
//   2. The E-th smallest key is found either by E rounds of a block-wide
//      minimum over keys above the previous one (small E, the steady state of
//      one eviction per step), or by an MSB-first radix select with 8-bit
//      digits and an LDS histogram (large E, e.g. the first eviction).
//   3. Evicted slots below `budget` are holes; kept slots at or above it are
//      movers.  A block-wide scan ranks both in slot order and the k-th mover
//      fills the k-th hole.  Sources and destinations are disjoint, so the
//      moves need no ordering among themselves.
//   4. score / pos move in the same kernel; K / V rows move in the same kernel
//      when there are few of them, otherwise in a grid-wide copy kernel.
//   5. Optional: the kept positions, ascending, via an LDS bitmap over positions.
// When the layer has at most 16384 slots and at most 256 of them move (the
// steady state of one eviction per step, and most first evictions), the keys
// are computed once into LDS with one coalesced pass over score and pos, and
// the selection, the classification and the move lists all stay in LDS: the
// only other global round trip is the moved rows themselves.
#include <algorithm>
#include <type_traits>

#include "vz_internal.h"

namespace {

constexpr int kSel = 1024;
constexpr int kSelWaves = kSel / vz::kWave;
constexpr int kSmallE = 8;        // up to this many evictions: rounds of block minima
constexpr int kInlineRows = 256;  // up to this many moved slots: K/V copied by the select block
constexpr int kBitmapWords = 8192;  // kept-position bitmap: 2^18 positions
constexpr int kLdsSlots = 16384;    // slots whose keys fit in LDS
constexpr uint64_t kNoKey = ~0ull;  // LDS key of a slot that does not compete
constexpr int kFoldSlots = 9 * kSel;  // slots the fused fold + select kernel takes

// Block-shared state of the select kernels.  KEYS: the rank keys of the
// layer's slots fit in LDS (kNoKey for sinks and recent slots); the
// kept-position bitmap then aliases the key array (free by the time the bitmap
// is built), otherwise it is an array of its own.
template <bool KEYS>
struct SelShared {
    uint64_t red64[kSelWaves];
    int red_a[kSelWaves];
    int red_b[kSelWaves];
    uint32_t hist[256];
    uint64_t prefix;
    int krem;
    int cnt;
    int32_t ev[kSmallE];     // slots of the evicted keys found by the rounds (keys in LDS only)
    int32_t holes[kSmallE];  // those below the budget, ascending
    int nm;
    float pre_a[kSmallE];    // fused fold: new score and position of the slots at or past the budget
    int32_t pre_p[kSmallE];
    int32_t src[kInlineRows], dst[kInlineRows];  // move lists (keys in LDS only)
    uint64_t keys[KEYS ? kLdsSlots : 1];
    uint32_t own_bitmap[KEYS ? 1 : kBitmapWords];
    __device__ uint32_t* bitmap() { return KEYS ? reinterpret_cast<uint32_t*>(keys) : own_bitmap; }
};
static_assert(kLdsSlots * 2 >= kBitmapWords, "the key array holds the bitmap");

template <class SH>
__device__ uint64_t block_min_u64(uint64_t v, SH& sh) {
    v = vz::wave_min_u64(v);
    const int w = threadIdx.x / vz::kWave;
    __syncthreads();
    if ((threadIdx.x % vz::kWave) == 0) sh.red64[w] = v;
    __syncthreads();
    uint64_t r = sh.red64[0];
    for (int i = 1; i < kSelWaves; ++i) r = sh.red64[i] < r ? sh.red64[i] : r;
    return r;
}

// Inclusive wave scan of an int.
__device__ __forceinline__ int wave_incl_scan(int v) {
    const int lane = threadIdx.x % vz::kWave;
#pragma unroll
    for (int o = 1; o < vz::kWave; o <<= 1) {
        int t = __shfl_up(v, o, vz::kWave);
        if (lane >= o) v += t;
    }
    return v;
}

// Exclusive block scan of two ints; also returns the block totals.
template <class SH>
__device__ void block_scan2(int a, int b, int& ax, int& bx, int& at, int& bt, SH& sh) {
    const int ia = wave_incl_scan(a), ib = wave_incl_scan(b);
    const int w = threadIdx.x / vz::kWave, lane = threadIdx.x % vz::kWave;
    __syncthreads();
    if (lane == vz::kWave - 1) {
        sh.red_a[w] = ia;
        sh.red_b[w] = ib;
    }
    __syncthreads();
    int pa = 0, pb = 0, ta = 0, tb = 0;
    for (int i = 0; i < kSelWaves; ++i) {
        if (i < w) {
            pa += sh.red_a[i];
            pb += sh.red_b[i];
        }
        ta += sh.red_a[i];
        tb += sh.red_b[i];
    }
    ax = pa + ia - a;
    bx = pb + ib - b;
    at = ta;
    bt = tb;
}

// One layer of one sequence: the slots of its planes start at A, P (score,
// position) and k0, v0 (row 0 of KV head 0; head h is head_stride elements
// further).  src_g / dst_g: global move lists (used when LK is false);
// n_out: receives the number of moves left for the copy kernel; kept: NULL or
// the layer's kept-position output.
template <class T>
struct SelJob {
    float* A;
    int32_t* P;
    T* k0;
    T* v0;
    size_t head_stride;
    int32_t* src_g;
    int32_t* dst_g;
    int32_t* n_out;
    int32_t* kept;
    int32_t len, budget, n_sink, M, next_pos, Hkv;
    int inline_kv;
    // READY callers: this thread's smallest competing key and its slot
    // (~0 and -1 without one), which the first minimum round uses instead of
    // reading the keys back
    uint64_t first_best;
    int32_t first_best_j;
};

// LK: this layer's keys are kept in LDS (needs sh.keys and len <= kLdsSlots
// and inline_kv).  READY: the caller has already filled sh.keys (and passed a
// barrier) and passes each thread's smallest key; only with LK.  With one
// eviction the keys are never read back, so such a caller may leave them out.
// move_fn(n_moves, src, dst), when given, may perform the moves itself (and
// return true) instead of the copies below.
template <int DT, int D, bool LK, class SH, bool READY = false, class MoveFn = std::nullptr_t>
__device__ void select_body(const SelJob<typename vz::Elem<DT>::T>& job, SH& sh, MoveFn move_fn = nullptr) {
    using T = typename vz::Elem<DT>::T;
    constexpr int PER = vz::Elem<DT>::kPer16B;
    constexpr int CH = D / PER;
    uint64_t* const s_keys = sh.keys;
    uint32_t* const bitmap = sh.bitmap();
    int32_t* const s_src = sh.src;
    int32_t* const s_dst = sh.dst;
    int32_t* const s_ev = sh.ev;

    const int tid = threadIdx.x;
    float* A = job.A;
    int32_t* P = job.P;
    const int len = job.len, budget = job.budget, n_sink = job.n_sink, M = job.M, next_pos = job.next_pos;
    const int Hkv = job.Hkv;
    const int E = len > budget ? len - budget : 0;
    const int32_t recent_from = next_pos - M;
    auto is_mid = [&](int32_t p) { return p >= n_sink && p < recent_from; };
    if (LK && !READY) {
        // Every slot's key in one round: up to kLdsSlots / kSel slots per
        // thread, all loads issued before any use (indexes past the end are
        // clamped, so no load sits behind a branch).  8 per thread while they
        // suffice, 16 otherwise (e.g. 8193 slots would take a second round
        // trip at 8).
        auto load_keys = [&](auto per_thread) {
            constexpr int B = decltype(per_thread)::value;
            int32_t pv[B];
            float av[B];
#pragma unroll
            for (int b = 0; b < B; ++b) {
                // clamped into the slots: slot 0 exists even when len = 0 (cap >= 1)
                const int j = min(tid + b * kSel, max(len - 1, 0));
                pv[b] = P[j];
                av[b] = A[j];
            }
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int j = tid + b * kSel;
                if (j < len) s_keys[j] = is_mid(pv[b]) ? vz::rank_key(av[b], pv[b]) : kNoKey;
            }
        };
        static_assert(kLdsSlots == 16 * kSel, "one round of 16 keys per thread covers the LDS key array");
        if (len <= 8 * kSel)
            load_keys(std::integral_constant<int, 8>{});
        else
            load_keys(std::integral_constant<int, 16>{});
        __syncthreads();
    }
    // key of slot j and whether it competes
    auto key_at = [&](int j, uint64_t& k) -> bool {
        if (LK) {
            k = s_keys[j];
            return k != kNoKey;
        }
        const int32_t p = P[j];
        if (!is_mid(p)) return false;
        k = vz::rank_key(A[j], p);
        return true;
    };

    // ---- threshold: evict middle slots whose key >> shift <= thr >> shift ----
    uint64_t thr = 0;
    int shift = 0;
    if (E > 0 && E <= kSmallE) {
        uint64_t tau = 0;
        int found = 0;
        for (int r = 0; r < E; ++r) {
            uint64_t best = ~0ull;
            int best_j = -1;
            if (READY && r == 0) {
                best = job.first_best;
                best_j = job.first_best_j;
            } else {
                for (int j = tid; j < len; j += kSel) {
                    uint64_t k;
                    if (!key_at(j, k)) continue;
                    if (k > tau && k < best) {
                        best = k;
                        best_j = j;
                    }
                }
            }
            tau = block_min_u64(best, sh);
            if (tau == ~0ull) break;  // fewer middle slots than E
            // keys are distinct (they hold the position), so one thread owns the minimum
            if (LK && best == tau) {
                s_ev[r] = best_j;
                if (E == 1) {
                    // one eviction: len = budget + 1, so slot `budget` is the only
                    // slot at or past the budget, and it moves into the hole
                    // unless it is the evicted one
                    sh.nm = best_j < budget ? 1 : 0;
                    s_src[0] = budget;
                    s_dst[0] = best_j;
                }
            }
            ++found;
        }
        thr = tau;
        shift = 0;
        if (LK && E == 1 && found == 1) {
            __syncthreads();  // the pair the minimum's owner wrote
        } else if (LK) {
            // Holes: evicted slots below the budget; movers: kept slots at or
            // above it; the k-th mover fills the k-th hole, both in slot order
            // (at most kSmallE of each, so one thread pairs them).
            __syncthreads();
            if (tid == 0) {
                int32_t* const holes = sh.holes;  // in LDS: indexed at run time without scratch memory
                int nh = 0;
                for (int r = 0; r < found; ++r)
                    if (s_ev[r] < budget) holes[nh++] = s_ev[r];
                for (int a = 1; a < nh; ++a)  // ascending slots
                    for (int b = a; b > 0 && holes[b - 1] > holes[b]; --b) {
                        const int t = holes[b];
                        holes[b] = holes[b - 1];
                        holes[b - 1] = t;
                    }
                int nm = 0;
                for (int j = budget; j < len && nm < nh; ++j) {
                    bool ev = false;
                    for (int r = 0; r < found; ++r) ev = ev || s_ev[r] == j;
                    if (!ev) {
                        s_src[nm] = j;
                        s_dst[nm] = holes[nm];
                        ++nm;
                    }
                }
                sh.nm = nm;
            }
            __syncthreads();
        }
    } else if (E > kSmallE) {
        uint64_t prefix = 0;
        int krem = E;
        for (int s = 56;; s -= 8) {
            if (tid < 256) sh.hist[tid] = 0;
            __syncthreads();
            for (int j = tid; j < len; j += kSel) {
                uint64_t k;
                if (!key_at(j, k)) continue;
                if (s == 56 || (k >> (s + 8)) == (prefix >> (s + 8)))
                    atomicAdd(&sh.hist[(k >> s) & 255u], 1u);
            }
            __syncthreads();
            if (tid < vz::kWave) {  // wave 0 finds the bin holding the krem-th smallest candidate
                int c4[4], sum = 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    c4[i] = static_cast<int>(sh.hist[tid * 4 + i]);
                    sum += c4[i];
                }
                const int incl = wave_incl_scan(sum);
                const int excl = incl - sum;
                const bool hit = excl < krem && incl >= krem;
                const unsigned long long mask = __ballot(hit);
                if (mask == 0ull) {  // fewer candidates than E: take everything
                    if (tid == 0) {
                        sh.prefix = prefix | (255ull << s);
                        sh.krem = 0;
                        sh.cnt = 0;
                    }
                } else if (hit) {
                    int cum = excl, b = 3;
                    for (int i = 0; i < 4; ++i) {
                        if (cum + c4[i] >= krem) {
                            b = i;
                            break;
                        }
                        cum += c4[i];
                    }
                    sh.prefix = prefix | (static_cast<uint64_t>(tid * 4 + b) << s);
                    sh.krem = krem - cum;
                    sh.cnt = c4[b];
                }
            }
            __syncthreads();
            prefix = sh.prefix;
            krem = sh.krem;
            const int cnt = sh.cnt;
            if (cnt == krem || s == 0) {
                thr = prefix;
                shift = s;
                break;
            }
        }
    }

    // ---- holes (evicted, slot < budget) and movers (kept, slot >= budget) ----
    int32_t* src = LK ? s_src : job.src_g;
    int32_t* dst = LK ? s_dst : job.dst_g;
    int n_moves = 0;
    if (LK && E > 0 && E <= kSmallE) {
        n_moves = sh.nm;  // paired above
    } else {
        const int per = (len + kSel - 1) / kSel;
        const int j0 = min(tid * per, len), j1 = min(j0 + per, len);
        auto evicted = [&](int j) -> bool {
            if (E == 0) return false;
            uint64_t k;
            if (!key_at(j, k)) return false;
            return (k >> shift) <= (thr >> shift);
        };
        int nh = 0, nm = 0;
        for (int j = j0; j < j1; ++j) {
            const bool ev = evicted(j);
            if (j < budget) nh += ev ? 1 : 0;
            else nm += ev ? 0 : 1;
        }
        int hx, mx, ht, mt;
        block_scan2(nh, nm, hx, mx, ht, mt, sh);
        for (int j = j0; j < j1; ++j) {
            const bool ev = evicted(j);
            if (j < budget) {
                if (ev) dst[hx++] = j;
            } else if (!ev) {
                src[mx++] = j;
            }
        }
        n_moves = min(ht, mt);
        __syncthreads();
    }

    bool moved = false;
    if constexpr (!std::is_same<MoveFn, std::nullptr_t>::value) moved = move_fn(n_moves, src, dst);
    if (!moved)
        for (int r = tid; r < n_moves; r += kSel) {
            const int s = src[r], d = dst[r];
            A[d] = A[s];
            P[d] = P[s];
        }
    if (tid == 0) *job.n_out = (LK || job.inline_kv) ? 0 : n_moves;
    if (!moved && (LK || job.inline_kv)) {
        const int total = n_moves * Hkv * 2 * CH;
        for (int i = tid; i < total; i += kSel) {
            const int c = i % CH;
            int t = i / CH;
            const int which = t & 1;
            t >>= 1;
            const int h = t % Hkv, r = t / Hkv;
            T* base = (which ? job.v0 : job.k0) + h * job.head_stride + c * PER;
            *reinterpret_cast<uint4*>(base + static_cast<size_t>(dst[r]) * D) =
                *reinterpret_cast<const uint4*>(base + static_cast<size_t>(src[r]) * D);
        }
    }

    if (job.kept) {
        __syncthreads();
        const int new_len = E > 0 ? budget : len;
        const int words = (next_pos + 31) / 32;
        for (int w = tid; w < words; w += kSel) bitmap[w] = 0u;
        __syncthreads();
        for (int j = tid; j < new_len; j += kSel) {
            const int32_t p = P[j];
            if (p >= 0 && p < next_pos) atomicOr(&bitmap[p >> 5], 1u << (p & 31));
        }
        __syncthreads();
        const int wpt = (words + kSel - 1) / kSel;
        const int w0 = min(tid * wpt, words), w1 = min(w0 + wpt, words);
        int c = 0;
        for (int w = w0; w < w1; ++w) c += __popc(bitmap[w]);
        int cx, dummy, ct, dt;
        block_scan2(c, 0, cx, dummy, ct, dt, sh);
        int32_t* outp = job.kept;
        for (int w = w0; w < w1; ++w) {
            uint32_t bits = bitmap[w];
            while (bits) {
                const int b = __ffs(bits) - 1;
                bits &= bits - 1;
                if (cx < budget) outp[cx] = w * 32 + b;
                ++cx;
            }
        }
    }
}

// Single sequence: one block per layer.
template <int DT, int D, bool LK>
__global__ __launch_bounds__(kSel) void select_kernel(const VzEvictArgs a, int32_t M, int32_t* __restrict__ ws_n,
                                                      int32_t* __restrict__ ws_src, int32_t* __restrict__ ws_dst,
                                                      int inline_kv) {
    using T = typename vz::Elem<DT>::T;
    __shared__ SelShared<LK> sh;
    const int l = blockIdx.x;
    const size_t row = static_cast<size_t>(l) * a.cap;
    SelJob<T> job;
    job.A = a.score + row;
    job.P = a.pos + row;
    job.k0 = static_cast<T*>(a.k_cache) + row * a.Hkv * D;
    job.v0 = static_cast<T*>(a.v_cache) + row * a.Hkv * D;
    job.head_stride = static_cast<size_t>(a.cap) * D;
    job.src_g = ws_src + row;
    job.dst_g = ws_dst + row;
    job.n_out = ws_n + l;
    job.kept = a.kept_pos_out ? a.kept_pos_out + static_cast<size_t>(l) * a.budget : nullptr;
    job.len = a.len;
    job.budget = a.budget;
    job.n_sink = a.n_sink;
    job.M = M;
    job.next_pos = a.next_pos;
    job.Hkv = a.Hkv;
    job.inline_kv = inline_kv;
    select_body<DT, D, LK>(job, sh);
}

// Decode step's score fold (Sec. 3.2.2 Eq. 6) fused with the eviction that
// follows it, one block per layer: every slot's new score is formed from the
// old score and the KV heads' head-group sums a whole-range decode kernel
// left in the workspace (the same additions in the same order as the
// separate fold kernel: A = gamma A + ((S_0 + S_1) + ...) with the zero pad for
// the new slot), stored, and turned into its rank key in LDS directly, so the
// selection starts without re-reading the scores.  a.len and a.next_pos are
// the eviction's (after the append).
struct FoldIn {
    const float* sums;  // [L][NW][row]
    int64_t row;
    float gamma;
};

template <int DT, int D, int NW>
__global__ __launch_bounds__(kSel) void fold_select_kernel(const VzEvictArgs a, int32_t M, FoldIn f,
                                                           int32_t* __restrict__ ws_n) {
    using T = typename vz::Elem<DT>::T;
    __shared__ SelShared<true> sh;
    const int l = blockIdx.x, tid = threadIdx.x;
    const size_t row = static_cast<size_t>(l) * a.cap;
    float* const A = a.score + row;
    int32_t* const P = a.pos + row;
    const float* const S = f.sums + static_cast<size_t>(l) * NW * f.row;
    const int len = a.len;  // keys after the append; slot len - 1 is the new one
    const int32_t recent_from = a.next_pos - M;
    T* const k0 = static_cast<T*>(a.k_cache) + row * a.Hkv * D;
    T* const v0 = static_cast<T*>(a.v_cache) + row * a.Hkv * D;
    const size_t head_stride = static_cast<size_t>(a.cap) * D;
    // With at most kSmallE evictions the movers are among the E slots at or
    // past the budget: their K/V rows are loaded now, beside the fold's loads
    // (one 16-byte piece per thread), and their new score and position kept
    // in LDS, so that the moves after the selection are stores only.
    constexpr int PER = vz::Elem<DT>::kPer16B;
    constexpr int CH = D / PER;
    const int E = len > a.budget ? len - a.budget : 0;
    const bool pre = E > 0 && E <= kSmallE;
    const int n_pre = pre ? E * NW * 2 * CH : 0;
    static_assert(kSmallE * NW * 2 * CH <= kSel, "one piece per thread");
    uint4 piece = make_uint4(0, 0, 0, 0);
    int piece_slot = -1;
    T* piece_base = nullptr;
    if (tid < n_pre) {
        const int c = tid % CH;
        int t = tid / CH;
        const int which = t & 1;
        t >>= 1;
        const int h = t % NW;
        piece_slot = a.budget + t / NW;
        piece_base = (which ? v0 : k0) + h * head_stride + c * PER;
        piece = *reinterpret_cast<const uint4*>(piece_base + static_cast<size_t>(piece_slot) * D);
    }
    // the keys go to LDS only for the later minimum rounds (E >= 2) and the
    // radix select; the first round takes each thread's smallest key
    const bool keys_to_lds = E >= 2;
    uint64_t my_best = ~0ull;
    int my_best_j = -1;
    auto fold_keys = [&](auto per_thread) {
        constexpr int B = decltype(per_thread)::value;
        int32_t pv[B];
        float av[B], sv[B][NW];
#pragma unroll
        for (int b = 0; b < B; ++b) {  // every load issued before any use; indexes clamped
            const int j = min(tid + b * kSel, len - 1);
            pv[b] = P[j];
            av[b] = A[j];
#pragma unroll
            for (int g = 0; g < NW; ++g) sv[b][g] = S[g * f.row + j];
        }
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int j = tid + b * kSel;
            if (j < len) {
                float acc = sv[b][0];
#pragma unroll
                for (int g = 1; g < NW; ++g) acc += sv[b][g];
                const float a_new = fmaf(f.gamma, j < len - 1 ? av[b] : 0.f, acc);
                A[j] = a_new;
                const int32_t p = pv[b];
                const uint64_t key = p >= a.n_sink && p < recent_from ? vz::rank_key(a_new, p) : kNoKey;
                if (keys_to_lds) sh.keys[j] = key;
                if (key < my_best) {  // kNoKey never wins: keys hold the position, so they are below ~0
                    my_best = key;
                    my_best_j = j;
                }
                if (pre && j >= a.budget) {
                    sh.pre_a[j - a.budget] = a_new;
                    sh.pre_p[j - a.budget] = p;
                }
            }
        }
    };
    // 8 slots per thread, or 9 (up to kFoldSlots): one round of loads either way
    if (len <= 8 * kSel)
        fold_keys(std::integral_constant<int, 8>{});
    else
        fold_keys(std::integral_constant<int, 9>{});
    __syncthreads();  // keys in LDS; new scores visible to the block
    if (E == 0 && a.kept_pos_out == nullptr) return;
    SelJob<T> job;
    job.A = A;
    job.P = P;
    job.k0 = k0;
    job.v0 = v0;
    job.head_stride = head_stride;
    job.src_g = nullptr;
    job.dst_g = nullptr;
    job.n_out = ws_n + l;
    job.kept = a.kept_pos_out ? a.kept_pos_out + static_cast<size_t>(l) * a.budget : nullptr;
    job.len = len;
    job.budget = a.budget;
    job.n_sink = a.n_sink;
    job.M = M;
    job.next_pos = a.next_pos;
    job.Hkv = a.Hkv;
    job.inline_kv = 1;
    job.first_best = my_best;
    job.first_best_j = my_best_j;
    // the moves from the prefetched rows (pairs in LDS, at most kSmallE)
    auto move_pre = [&](int n_moves, const int32_t* src, const int32_t* dst) -> bool {
        if (!pre) return false;
        if (tid < n_moves) {
            const int sj = src[tid] - a.budget;
            A[dst[tid]] = sh.pre_a[sj];
            P[dst[tid]] = sh.pre_p[sj];
        }
        if (piece_slot >= 0)
            for (int r = 0; r < n_moves; ++r)
                if (src[r] == piece_slot)
                    *reinterpret_cast<uint4*>(piece_base + static_cast<size_t>(dst[r]) * D) = piece;
        return true;
    };
    select_body<DT, D, true, SelShared<true>, true>(job, sh, move_pre);
}

// Status of sequence s for an eviction (VZ_OK when it can be served).
__device__ int ragged_evict_status(const VzRagged& r, int s, int n_sink, int n_recent, bool kept) {
    const int64_t b = r.base[s];
    const int c = r.cap[s], n = r.len[s], B = r.budget[s], p = r.next_pos[s];
    if (n < 0 || c < 1 || b < 0 || b > r.total - c) return VZ_ERR_INVALID;
    if (n > c) return VZ_ERR_CAPACITY;
    const int M = n_recent < 0 ? B / 5 : n_recent;
    if (B < 1 || static_cast<int64_t>(n_sink) + M > B || p < n) return VZ_ERR_INVALID;
    if (kept && p > (1 << 18)) return VZ_ERR_UNSUPPORTED;
    return VZ_OK;
}

// Ragged batch: one block per (layer, sequence).  The keys go to LDS when the
// sequence's slots fit and few rows move, as in the single-sequence launch;
// every block leaves its copy-kernel count in ws_n (0 when nothing is left).
template <int DT, int D>
__global__ __launch_bounds__(kSel) void select_ragged_kernel(const VzEvictArgs a, int32_t* __restrict__ ws_n,
                                                             int32_t* __restrict__ ws_src,
                                                             int32_t* __restrict__ ws_dst) {
    using T = typename vz::Elem<DT>::T;
    __shared__ SelShared<true> sh;
    const int l = blockIdx.x, s = blockIdx.y;
    const VzRagged& r = a.rag;
    int32_t* const n_out = ws_n + static_cast<size_t>(s) * a.L + l;
    const int st = ragged_evict_status(r, s, a.n_sink, a.n_recent, a.kept_pos_out != nullptr);
    if (l == 0 && threadIdx.x == 0) {
        if (r.status) r.status[s] = st;
        if (a.new_len_out) {
            const int n = r.len[s], B = r.budget[s];
            a.new_len_out[s] = st == VZ_OK && n > B ? B : n;
        }
    }
    if (st != VZ_OK) {
        if (threadIdx.x == 0) *n_out = 0;
        return;
    }
    const int len = r.len[s], budget = r.budget[s];
    const int E = len > budget ? len - budget : 0;
    if (E == 0 && a.kept_pos_out == nullptr) {
        if (threadIdx.x == 0) *n_out = 0;
        return;
    }
    const size_t row = static_cast<size_t>(l) * r.total + r.base[s];
    SelJob<T> job;
    job.A = a.score + row;
    job.P = a.pos + row;
    job.k0 = static_cast<T*>(a.k_cache) + (static_cast<size_t>(l) * a.Hkv * r.total + r.base[s]) * D;
    job.v0 = static_cast<T*>(a.v_cache) + (static_cast<size_t>(l) * a.Hkv * r.total + r.base[s]) * D;
    job.head_stride = static_cast<size_t>(r.total) * D;
    job.src_g = ws_src + row;
    job.dst_g = ws_dst + row;
    job.n_out = n_out;
    job.kept = a.kept_pos_out ? a.kept_pos_out + row : nullptr;
    job.len = len;
    job.budget = budget;
    job.n_sink = a.n_sink;
    job.M = a.n_recent < 0 ? budget / 5 : a.n_recent;
    job.next_pos = r.next_pos[s];
    job.Hkv = a.Hkv;
    job.inline_kv = E <= kInlineRows ? 1 : 0;
    if (job.inline_kv && len <= kLdsSlots)
        select_body<DT, D, true>(job, sh);
    else
        select_body<DT, D, false>(job, sh);
}

// Copy kernel for layers with many moved rows: grid (jobs, y); job x =
// (sequence, layer) (the layer alone for a single sequence), whose gridDim.y
// blocks split its moves.
template <int DT, int D, bool RAG>
__global__ __launch_bounds__(256) void compact_kernel(const VzEvictArgs a, const int32_t* __restrict__ ws_n,
                                                      const int32_t* __restrict__ ws_src,
                                                      const int32_t* __restrict__ ws_dst) {
    using T = typename vz::Elem<DT>::T;
    constexpr int PER = vz::Elem<DT>::kPer16B;
    constexpr int CH = D / PER;
    const int job = blockIdx.x;
    const int n = ws_n[job];
    if (n == 0) return;
    const int l = RAG ? job % a.L : job;
    const int64_t plane = RAG ? a.rag.total : a.cap;
    const int64_t base = RAG ? a.rag.base[job / a.L] : 0;
    const size_t row = static_cast<size_t>(l) * plane + base;
    const int32_t* src = ws_src + row;
    const int32_t* dst = ws_dst + row;
    const int64_t total = static_cast<int64_t>(n) * a.Hkv * 2 * CH;
    for (int64_t i = static_cast<int64_t>(blockIdx.y) * 256 + threadIdx.x; i < total;
         i += static_cast<int64_t>(gridDim.y) * 256) {
        const int c = static_cast<int>(i % CH);
        int64_t t = i / CH;
        const int which = static_cast<int>(t & 1);
        t >>= 1;
        const int h = static_cast<int>(t % a.Hkv);
        const int r = static_cast<int>(t / a.Hkv);
        T* hb = static_cast<T*>(which ? a.v_cache : a.k_cache) +
                ((static_cast<size_t>(l) * a.Hkv + h) * plane + base) * D + c * PER;
        *reinterpret_cast<uint4*>(hb + static_cast<size_t>(dst[r]) * D) =
            *reinterpret_cast<const uint4*>(hb + static_cast<size_t>(src[r]) * D);
    }
}

// Workspace: move counts [jobs rounded up to 64], then source and destination
// lists [L][plane] each.
struct EvictWs {
    int32_t* n;
    int32_t* src;
    int32_t* dst;
    EvictWs(void* ws, int64_t jobs, int32_t L, int64_t plane) {
        n = static_cast<int32_t*>(ws);
        src = n + 64 * ((jobs + 63) / 64);
        dst = src + static_cast<size_t>(L) * plane;
    }
};

template <int DT, int D>
hipError_t launch(const VzEvictArgs& a, hipStream_t stream) {
    constexpr int CH = D / vz::Elem<DT>::kPer16B;
    if (a.rag.n > 0) {
        const int64_t jobs = static_cast<int64_t>(a.rag.n) * a.L;
        EvictWs w(a.ws, jobs, a.L, a.rag.total);
        hipLaunchKernelGGL((select_ragged_kernel<DT, D>), dim3(a.L, a.rag.n), dim3(kSel), 0, stream, a, w.n, w.src,
                           w.dst);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        // most jobs move their rows in the select block and leave 0 here
        const int gy = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(64, 4096 / jobs)));
        hipLaunchKernelGGL((compact_kernel<DT, D, true>), dim3(static_cast<unsigned>(jobs), gy), dim3(256), 0,
                           stream, a, w.n, w.src, w.dst);
        return hipGetLastError();
    }
    const int E = a.len > a.budget ? a.len - a.budget : 0;
    if (E == 0 && a.kept_pos_out == nullptr) return hipSuccess;
    EvictWs w(a.ws, a.L, a.L, a.cap);
    const int M = a.n_recent < 0 ? a.budget / 5 : a.n_recent;
    const int inline_kv = E <= kInlineRows ? 1 : 0;
    if (inline_kv && a.len <= kLdsSlots)
        hipLaunchKernelGGL((select_kernel<DT, D, true>), dim3(a.L), dim3(kSel), 0, stream, a, M, w.n, w.src, w.dst,
                           inline_kv);
    else
        hipLaunchKernelGGL((select_kernel<DT, D, false>), dim3(a.L), dim3(kSel), 0, stream, a, M, w.n, w.src, w.dst,
                           inline_kv);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || inline_kv) return e;
    const int64_t chunks = static_cast<int64_t>(E) * a.Hkv * 2 * CH;
    const int gy = static_cast<int>(std::min<int64_t>((chunks + 255) / 256, 2048));
    hipLaunchKernelGGL((compact_kernel<DT, D, false>), dim3(a.L, gy), dim3(256), 0, stream, a, w.n, w.src, w.dst);
    return hipGetLastError();
}

template <int DT, int D, int NW>
hipError_t launch_fold(const VzEvictArgs& a, const float* sums, int64_t row, float gamma, hipStream_t stream) {
    EvictWs w(a.ws, a.L, a.L, a.cap);
    const int M = a.n_recent < 0 ? a.budget / 5 : a.n_recent;
    hipLaunchKernelGGL((fold_select_kernel<DT, D, NW>), dim3(a.L), dim3(kSel), 0, stream, a, M,
                       FoldIn{sums, row, gamma}, w.n);
    return hipGetLastError();
}

}  // namespace

size_t vz_evict_ws_bytes(int32_t L, int64_t plane, int32_t n_seqs) {
    const int64_t jobs = static_cast<int64_t>(n_seqs > 0 ? n_seqs : 1) * L;
    return (static_cast<size_t>(64) * ((jobs + 63) / 64) + 2 * static_cast<size_t>(L) * plane) * sizeof(int32_t);
}

hipError_t vz_launch_evict(const VzEvictArgs& a, hipStream_t stream) {
    if (a.dtype == VZ_BF16 && a.d == 128) return launch<VZ_BF16, 128>(a, stream);
    if (a.dtype == VZ_BF16 && a.d == 64) return launch<VZ_BF16, 64>(a, stream);
    if (a.dtype == VZ_F32 && a.d == 128) return launch<VZ_F32, 128>(a, stream);
    if (a.dtype == VZ_F32 && a.d == 64) return launch<VZ_F32, 64>(a, stream);
    return hipErrorInvalidValue;
}

bool vz_fold_evict_ok(int32_t dtype, int32_t d, int32_t Hkv, int32_t len, int32_t budget) {
    const int E = len > budget ? len - budget : 0;
    return dtype == VZ_BF16 && d == 128 && (Hkv == 1 || Hkv == 2 || Hkv == 4) && len <= kFoldSlots &&
           E <= kInlineRows;
}

hipError_t vz_launch_fold_evict(const VzEvictArgs& a, const float* sums, int64_t row, float gamma,
                                hipStream_t stream) {
    switch (a.Hkv) {
        case 1: return launch_fold<VZ_BF16, 128, 1>(a, sums, row, gamma, stream);
        case 2: return launch_fold<VZ_BF16, 128, 2>(a, sums, row, gamma, stream);
        case 4: return launch_fold<VZ_BF16, 128, 4>(a, sums, row, gamma, stream);
        default: return hipErrorInvalidValue;
    }
}
