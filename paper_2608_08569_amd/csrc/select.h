// Stage-2 selection (Sec. 3.2.2, Eq. 7-9) for one layer of one sequence, run
// by a whole block of NT threads, and the score fold of Eq. (6) fused in front
// of it.  Shared by the eviction kernels (evict.hip, 1024-thread blocks) and
// the whole-range decode kernel (decode_range.hip), whose last-arriving
// workgroup of each layer folds the scores and selects with its 512 threads.
//
//   1. Rank key per slot: (order-preserving score bits << 32) | ~pos, so the
//      larger key is the more important slot (ties to the smaller position).
//      Only middle slots (not sink, not recent) compete.  E = len - budget of
//      them are evicted: the E smallest keys.
//   2. The E-th smallest key is found either by E rounds of a block-wide
//      minimum over keys above the previous one (small E, the steady state of
//      one eviction per step), or by an MSB-first radix select with 8-bit
//      digits and an LDS histogram (large E, e.g. the first eviction).
//   3. Evicted slots below `budget` are holes; kept slots at or above it are
//      movers.  The k-th mover fills the k-th hole, both in slot order.
//      Sources and destinations are disjoint, so the moves need no ordering
//      among themselves.
//   4. score / pos move in the same block; K / V rows move in the same block
//      when there are few of them, otherwise in a grid-wide copy kernel.
//   5. Optional: the kept positions, ascending, via an LDS bitmap over positions.
#pragma once

#include <type_traits>

#include "vz_internal.h"

namespace vz_sel {

constexpr int kSmallE = 8;          // up to this many evictions: rounds of block minima
constexpr int kInlineRows = 256;    // up to this many moved slots: K/V copied by the select block
constexpr int kBitmapWords = 8192;  // kept-position bitmap: 2^18 positions
constexpr uint64_t kNoKey = ~0ull;  // LDS key of a slot that does not compete

// Block-shared state of a selection by NT threads.  NKEYS > 0: the rank keys
// of up to NKEYS slots live in LDS (kNoKey for sinks and recent slots), and
// the kept-position bitmap aliases the key array (free by the time the bitmap
// is built); NKEYS = 0: keys are recomputed from memory and the bitmap is an
// array of its own.
template <int NT, int NKEYS>
struct SelShared {
    static constexpr int kKeys = NKEYS;
    static_assert(NKEYS == 0 || 2 * NKEYS >= kBitmapWords, "the key array holds the bitmap");
    uint64_t red64[NT / vz::kWave];
    int red_a[NT / vz::kWave];
    int red_b[NT / vz::kWave];
    uint32_t hist[256];
    uint64_t prefix;
    int krem;
    int cnt;
    int32_t ev[kSmallE];     // slots of the evicted keys found by the rounds (keys in LDS only)
    int32_t holes[kSmallE];  // those below the budget, ascending
    int nm;
    int32_t src[kInlineRows], dst[kInlineRows];  // move lists (keys in LDS only)
    uint64_t keys[NKEYS > 0 ? NKEYS : 1];
    uint32_t own_bitmap[NKEYS > 0 ? 1 : kBitmapWords];
    __device__ uint32_t* bitmap() { return NKEYS > 0 ? reinterpret_cast<uint32_t*>(keys) : own_bitmap; }
};

// A block barrier that orders LDS accesses only: unlike __syncthreads it does
// not wait for the block's outstanding global stores, so a selection can run
// while the scores the block just stored drain to memory.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int NT, class SH>
__device__ uint64_t block_min_u64(uint64_t v, SH& sh) {
    v = vz::wave_min_u64(v);
    const int w = threadIdx.x / vz::kWave;
    lds_barrier();
    if ((threadIdx.x % vz::kWave) == 0) sh.red64[w] = v;
    lds_barrier();
    uint64_t r = sh.red64[0];
    for (int i = 1; i < NT / vz::kWave; ++i) r = sh.red64[i] < r ? sh.red64[i] : r;
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
template <int NT, class SH>
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
    for (int i = 0; i < NT / vz::kWave; ++i) {
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
template <int NT, int DT, int D, bool LK, class SH, bool READY = false, class MoveFn = std::nullptr_t>
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
    if constexpr (LK && !READY) {
        // Every slot's key in one round: up to SH::kKeys / NT slots per
        // thread, all loads issued before any use (indexes past the end are
        // clamped, so no load sits behind a branch).  Half of that while it
        // suffices, all of it otherwise (e.g. 8193 slots would take a second
        // round trip at 8 of 1024 threads).
        auto load_keys = [&](auto per_thread) {
            constexpr int B = decltype(per_thread)::value;
            int32_t pv[B];
            float av[B];
#pragma unroll
            for (int b = 0; b < B; ++b) {
                // clamped into the slots: slot 0 exists even when len = 0 (cap >= 1)
                const int j = min(tid + b * NT, max(len - 1, 0));
                pv[b] = P[j];
                av[b] = A[j];
            }
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int j = tid + b * NT;
                if (j < len) s_keys[j] = is_mid(pv[b]) ? vz::rank_key(av[b], pv[b]) : kNoKey;
            }
        };
        constexpr int KPT = SH::kKeys / NT;
        static_assert(KPT * NT == SH::kKeys && KPT % 2 == 0, "one round covers the LDS key array");
        if (len <= KPT / 2 * NT)
            load_keys(std::integral_constant<int, KPT / 2>{});
        else
            load_keys(std::integral_constant<int, KPT>{});
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
                for (int j = tid; j < len; j += NT) {
                    uint64_t k;
                    if (!key_at(j, k)) continue;
                    if (k > tau && k < best) {
                        best = k;
                        best_j = j;
                    }
                }
            }
            tau = block_min_u64<NT>(best, sh);
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
            lds_barrier();  // the pair the minimum's owner wrote
        } else if (LK) {
            // Holes: evicted slots below the budget; movers: kept slots at or
            // above it; the k-th mover fills the k-th hole, both in slot order
            // (at most kSmallE of each, so one thread pairs them).
            lds_barrier();
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
            lds_barrier();
        }
    } else if (E > kSmallE) {
        uint64_t prefix = 0;
        int krem = E;
        for (int s = 56;; s -= 8) {
            if (tid < 256) sh.hist[tid] = 0;
            __syncthreads();
            for (int j = tid; j < len; j += NT) {
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
                    // the first of the lane's 4 bins where the count reaches krem
                    // (fixed indexes only: no private array in scratch memory)
                    int cum = excl, b = -1, cum_b = 0, cnt_b = 0;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const bool take = b < 0 && cum + c4[i] >= krem;
                        b = take ? i : b;
                        cum_b = take ? cum : cum_b;
                        cnt_b = take ? c4[i] : cnt_b;
                        cum += c4[i];
                    }
                    if (b < 0) {  // not reached: the lane holds the krem-th candidate
                        b = 3;
                        cum_b = cum;
                        cnt_b = c4[3];
                    }
                    sh.prefix = prefix | (static_cast<uint64_t>(tid * 4 + b) << s);
                    sh.krem = krem - cum_b;
                    sh.cnt = cnt_b;
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
        const int per = (len + NT - 1) / NT;
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
        block_scan2<NT>(nh, nm, hx, mx, ht, mt, sh);
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
        for (int r = tid; r < n_moves; r += NT) {
            const int s = src[r], d = dst[r];
            A[d] = A[s];
            P[d] = P[s];
        }
    if (tid == 0) *job.n_out = (LK || job.inline_kv) ? 0 : n_moves;
    if (!moved && (LK || job.inline_kv)) {
        const int total = n_moves * Hkv * 2 * CH;
        for (int i = tid; i < total; i += NT) {
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
        for (int w = tid; w < words; w += NT) bitmap[w] = 0u;
        __syncthreads();
        for (int j = tid; j < new_len; j += NT) {
            const int32_t p = P[j];
            if (p >= 0 && p < next_pos) atomicOr(&bitmap[p >> 5], 1u << (p & 31));
        }
        __syncthreads();
        const int wpt = (words + NT - 1) / NT;
        const int w0 = min(tid * wpt, words), w1 = min(w0 + wpt, words);
        int c = 0;
        for (int w = w0; w < w1; ++w) c += __popc(bitmap[w]);
        int cx, dummy, ct, dt;
        block_scan2<NT>(c, 0, cx, dummy, ct, dt, sh);
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


// The fold of Eq. (6) for every slot of one layer, then (when `select`) the
// selection above, by the block of NT threads that finishes a layer's decode
// step.  The decode left, per KV head g, every key's sum over g's query heads
// of p_hj in S[g * row + j] (written by other workgroups of the running
// kernel with device-coherent stores, so read here with device-coherent
// loads); the new score is A = gamma A + ((S_0 + S_1) + ...), in that order,
// with the zero pad for the new slot len - 1, whose position next_pos - 1 is
// written here.  Each new score is stored and turned into the slot's rank key
// at once (kept in registers for the first minimum round, in LDS when E >= 2),
// so the selection starts without re-reading the scores.
//
// Two slot layouts: the sums are read as 16-byte vectors, four consecutive
// slots per thread (4 (tid + r NT) + i), added up and handed over through LDS
// to the layout of everything else, one slot per thread and round (tid + b NT),
// which keeps the old scores' and positions' 4-byte accesses coalesced (those
// rows have no 16-byte alignment).  The old scores and positions are loaded
// (fold_prefetch) before the block knows it finishes the layer, so only the
// sums' round trip follows the arrival.  Buffer descriptors bound every
// access: slots past the old ones read as 0 (the zero pad) and stores past
// len are dropped, with no index clamping or branches.
//
// With at most kSmallE evictions the movers are among the E slots at or past
// the budget: their K/V rows are loaded at the start and their new score and
// position kept in LDS, so that the moves after the selection are stores
// only.  The new slot's K/V rows are always taken from k_new / v_new (its
// cache rows were written by other workgroups of the running kernel).
template <class T>
struct FoldLayer {
    float* A;
    int32_t* P;
    T* k0;
    T* v0;               // row 0 of KV head 0 of the layer; head h is h * head_stride elements further
    size_t head_stride;
    const float* S;      // head-group sums of the layer, [NW][row]
    int64_t row;
    const T* k_new;      // [NW][D]: the new slot's K and V rows
    const T* v_new;
    int32_t len, budget, n_sink, M, next_pos;  // after the append (slot len - 1 is new)
    float gamma;
    int32_t* kept;       // NULL or [budget]
    int32_t* n_out;
    bool select;         // false: the fold alone
};

// The old scores and positions of a thread's slots tid + b NT, b < B.
template <int B>
struct FoldOld {
    float a[B];
    int32_t p[B];
};

constexpr int kBufferDword3 = 0x00020000;  // raw buffer descriptor word 3 (32-bit data format)
constexpr int kCoherent = 16;              // buffer access cache policy: device scope (sc1)

// Issues the loads of the old scores A and positions P of a layer of len
// slots after the append (the new slot and those past it read as 0).
template <int NT, int B>
__device__ __forceinline__ void fold_prefetch(float* A, int32_t* P, int len, FoldOld<B>& o) {
    const int tid = threadIdx.x;
    const int old = len - 1;  // slots holding a previous score and position
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(A, 0, old * 4, kBufferDword3);
    const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(P, 0, old * 4, kBufferDword3);
#pragma unroll
    for (int b = 0; b < B; ++b) {
        o.a[b] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ra, (tid + b * NT) * 4, 0, 0));
        o.p[b] = static_cast<int32_t>(__builtin_amdgcn_raw_buffer_load_b32(rp, (tid + b * NT) * 4, 0, 0));
    }
}

// s_acc: LDS scratch of at least 4 R NT + 2 NT floats.  B NT and 4 R NT cover len.
template <int NT, int B, int R, int DT, int D, int NW, class SH>
__device__ void fold_select_layer(const FoldLayer<typename vz::Elem<DT>::T>& f, const FoldOld<B>& o, float* s_acc,
                                  SH& sh) {
    using T = typename vz::Elem<DT>::T;
    constexpr int PER = vz::Elem<DT>::kPer16B;
    constexpr int CH = D / PER;
    constexpr int NPIECE = (kSmallE * NW * 2 * CH + NT - 1) / NT;  // 16-byte pieces of the movers per thread
    const int tid = threadIdx.x;
    float* const A = f.A;
    int32_t* const P = f.P;
    const int len = f.len;
    const int32_t new_pos = f.next_pos - 1;
    const int32_t recent_from = f.next_pos - f.M;
    const int E = f.select && len > f.budget ? len - f.budget : 0;
    const bool pre = E > 0 && E <= kSmallE;
    const int n_pre = pre ? E * NW * 2 * CH : 0;
    uint4 piece[NPIECE];
    int piece_slot[NPIECE];
    T* piece_base[NPIECE];
#pragma unroll
    for (int i = 0; i < NPIECE; ++i) {
        piece[i] = make_uint4(0, 0, 0, 0);
        piece_slot[i] = -1;
        piece_base[i] = nullptr;
        const int x = tid + i * NT;
        if (x < n_pre) {
            const int c = x % CH;
            int t = x / CH;
            const int which = t & 1;
            t >>= 1;
            const int h = t % NW;
            const int slot = f.budget + t / NW;
            piece_base[i] = (which ? f.v0 : f.k0) + h * f.head_stride + c * PER;
            const T* from = slot == len - 1 ? (which ? f.v_new : f.k_new) + h * D + c * PER
                                            : piece_base[i] + static_cast<size_t>(slot) * D;
            piece[i] = *reinterpret_cast<const uint4*>(from);
            piece_slot[i] = slot;
        }
    }
    // ---- the sums over the KV heads, in head order, four slots per thread ----
    {
        float4 acc[R];
#pragma unroll
        for (int g0 = 0; g0 < NW; g0 += 4) {  // at most 4 KV heads' loads in flight
            constexpr int GB = NW < 4 ? NW : 4;
            float4 v[GB][R];
#pragma unroll
            for (int gg = 0; gg < GB; ++gg) {
                const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                    const_cast<float*>(f.S + (g0 + gg) * f.row), 0, static_cast<int>(f.row) * 4, kBufferDword3);
#pragma unroll
                for (int r = 0; r < R; ++r)
                    v[gg][r] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                                              rs, (tid + r * NT) * 16, 0, kCoherent));
            }
#pragma unroll
            for (int gg = 0; gg < GB; ++gg)
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    if (g0 + gg == 0) {
                        acc[r] = v[gg][r];
                    } else {
                        acc[r].x += v[gg][r].x;
                        acc[r].y += v[gg][r].y;
                        acc[r].z += v[gg][r].z;
                        acc[r].w += v[gg][r].w;
                    }
                }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) *reinterpret_cast<float4*>(s_acc + 4 * (tid + r * NT)) = acc[r];
    }
    lds_barrier();
    // ---- Eq. (6) and the rank keys, one slot per thread and round ----
    // Branch-free: the keys go to LDS for every slot index the rounds cover
    // (kNoKey past len) when the selection needs them there (E >= 2; the
    // first minimum round takes each thread's smallest key from registers),
    // and the rounds that can hold slots at or past the budget (the movers
    // when E <= kSmallE) leave every new score in s_acc and every position in
    // s_pos, whole rounds at a time.
    static_assert(SH::kKeys >= B * NT, "a key for every slot index of the rounds");
    const bool keys_to_lds = E >= 2;
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(A, 0, len * 4, kBufferDword3);
    const int b_mov = pre ? f.budget / NT : B;  // first round holding a mover
    int32_t* const s_pos = reinterpret_cast<int32_t*>(s_acc + 4 * R * NT);  // [2 NT]: rounds b_mov, b_mov + 1
    uint64_t my_best = ~0ull;
    int my_best_j = -1;
    auto rounds = [&](auto keys) {
        constexpr bool KEYS = decltype(keys)::value;
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int j = tid + b * NT;
            const float a_new = fmaf(f.gamma, o.a[b], s_acc[j]);  // o.a is 0 for the new slot (zero pad)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, a_new), ra, j * 4, 0, 0);  // dropped past len
            const int32_t p = j == len - 1 ? new_pos : o.p[b];
            const bool mid = j < len && p >= f.n_sink && p < recent_from;
            const uint64_t key = mid ? vz::rank_key(a_new, p) : kNoKey;
            const bool better = key < my_best;  // kNoKey never wins: keys hold the position, so they are below ~0
            my_best = better ? key : my_best;
            my_best_j = better ? j : my_best_j;
            if constexpr (KEYS) sh.keys[j] = key;
            if (b == b_mov || b == b_mov + 1) {  // wave-uniform
                s_acc[j] = a_new;
                s_pos[j - b_mov * NT] = p;
            }
        }
    };
    if (keys_to_lds)
        rounds(std::true_type{});
    else
        rounds(std::false_type{});
    if (tid == (len - 1) % NT) P[len - 1] = new_pos;  // Eq. (1): the new slot's position
    lds_barrier();  // keys and movers in LDS (the scores' stores may still drain)
    if (!f.select || (E == 0 && f.kept == nullptr)) return;
    SelJob<T> job;
    job.A = A;
    job.P = P;
    job.k0 = f.k0;
    job.v0 = f.v0;
    job.head_stride = f.head_stride;
    job.src_g = nullptr;
    job.dst_g = nullptr;
    job.n_out = f.n_out;
    job.kept = f.kept;
    job.len = len;
    job.budget = f.budget;
    job.n_sink = f.n_sink;
    job.M = f.M;
    job.next_pos = f.next_pos;
    job.Hkv = NW;
    job.inline_kv = 1;
    job.first_best = my_best;
    job.first_best_j = my_best_j;
    // The moves, always done here: the new slot's K/V rows come from k_new /
    // v_new, its score and position from this block's own stores.
    auto move_rows = [&](int n_moves, const int32_t* src, const int32_t* dst) -> bool {
        if (pre) {  // from LDS and the prefetched rows (at most kSmallE)
            if (tid < n_moves) {
                A[dst[tid]] = s_acc[src[tid]];
                P[dst[tid]] = s_pos[src[tid] - b_mov * NT];
            }
#pragma unroll
            for (int i = 0; i < NPIECE; ++i)
                if (piece_slot[i] >= 0)
                    for (int r = 0; r < n_moves; ++r)
                        if (src[r] == piece_slot[i])
                            *reinterpret_cast<uint4*>(piece_base[i] + static_cast<size_t>(dst[r]) * D) = piece[i];
            return true;
        }
        __syncthreads();  // every new score and the new position stored (read back below)
        for (int r = tid; r < n_moves; r += NT) {
            A[dst[r]] = A[src[r]];
            P[dst[r]] = P[src[r]];
        }
        const int total = n_moves * NW * 2 * CH;
        for (int i = tid; i < total; i += NT) {
            const int c = i % CH;
            int t = i / CH;
            const int which = t & 1;
            t >>= 1;
            const int h = t % NW, r = t / NW;
            T* const base = (which ? f.v0 : f.k0) + h * f.head_stride + c * PER;
            const T* const from = src[r] == len - 1 ? (which ? f.v_new : f.k_new) + h * D + c * PER
                                                    : base + static_cast<size_t>(src[r]) * D;
            *reinterpret_cast<uint4*>(base + static_cast<size_t>(dst[r]) * D) = *reinterpret_cast<const uint4*>(from);
        }
        return true;
    };
    select_body<NT, DT, D, true, SH, true>(job, sh, move_rows);
}

}  // namespace vz_sel
