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

#include "vz_internal.h"

namespace {

constexpr int kSel = 1024;
constexpr int kSelWaves = kSel / vz::kWave;
constexpr int kSmallE = 8;        // up to this many evictions: rounds of block minima
constexpr int kInlineRows = 256;  // up to this many moved slots: K/V copied by the select block
constexpr int kBitmapWords = 8192;  // kept-position bitmap: 2^18 positions
constexpr int kLdsSlots = 16384;    // slots whose keys fit in LDS
constexpr uint64_t kNoKey = ~0ull;  // LDS key of a slot that does not compete

// Block-shared state; the kept-position bitmap is its own array unless the
// LDS key array (free by then) holds it.
template <bool OWN_BITMAP>
struct SelShared {
    uint64_t red64[kSelWaves];
    int red_a[kSelWaves];
    int red_b[kSelWaves];
    uint32_t hist[256];
    uint64_t prefix;
    int krem;
    int cnt;
    uint32_t bitmap[OWN_BITMAP ? kBitmapWords : 1];
};

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

template <int DT, int D, bool LK>
__global__ __launch_bounds__(kSel) void select_kernel(
    typename vz::Elem<DT>::T* __restrict__ k_cache, typename vz::Elem<DT>::T* __restrict__ v_cache,
    float* __restrict__ score, int32_t* __restrict__ pos, int32_t len, int32_t budget, int32_t n_sink,
    int32_t M, int32_t next_pos, int32_t* __restrict__ kept_pos_out, int32_t Hkv, int32_t cap,
    int32_t* __restrict__ ws_n, int32_t* __restrict__ ws_src, int32_t* __restrict__ ws_dst, int inline_kv) {
    using T = typename vz::Elem<DT>::T;
    constexpr int PER = vz::Elem<DT>::kPer16B;
    constexpr int CH = D / PER;
    __shared__ SelShared<!LK> sh;
    // LK: the rank keys of the layer's slots (kNoKey for sinks and recent
    // slots) and the move lists live in LDS
    __shared__ uint64_t s_keys[LK ? kLdsSlots : 1];
    static_assert(!LK || kLdsSlots * 2 >= kBitmapWords, "the key array holds the bitmap");
    uint32_t* const bitmap = LK ? reinterpret_cast<uint32_t*>(s_keys) : sh.bitmap;
    __shared__ int32_t s_src[LK ? kInlineRows : 1], s_dst[LK ? kInlineRows : 1];

    const int l = blockIdx.x;
    const int tid = threadIdx.x;
    float* A = score + static_cast<size_t>(l) * cap;
    int32_t* P = pos + static_cast<size_t>(l) * cap;
    const int E = len > budget ? len - budget : 0;
    const int32_t recent_from = next_pos - M;
    auto is_mid = [&](int32_t p) { return p >= n_sink && p < recent_from; };
    if (LK) {
        // 8 slots per thread and round, every load issued before any use (no
        // load behind a branch)
        constexpr int B = 8;
        for (int j0 = tid; j0 < len; j0 += B * kSel) {
            int32_t pv[B];
            float av[B];
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int j = min(j0 + b * kSel, len - 1);
                pv[b] = P[j];
                av[b] = A[j];
            }
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int j = j0 + b * kSel;
                if (j < len) s_keys[j] = is_mid(pv[b]) ? vz::rank_key(av[b], pv[b]) : kNoKey;
            }
        }
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
    // slots of the evicted keys, found by the rounds below (LK only)
    __shared__ int32_t s_ev[LK ? kSmallE : 1];
    __shared__ int s_nm;
    if (E > 0 && E <= kSmallE) {
        uint64_t tau = 0;
        int found = 0;
        for (int r = 0; r < E; ++r) {
            uint64_t best = ~0ull;
            int best_j = -1;
            for (int j = tid; j < len; j += kSel) {
                uint64_t k;
                if (!key_at(j, k)) continue;
                if (k > tau && k < best) {
                    best = k;
                    best_j = j;
                }
            }
            tau = block_min_u64(best, sh);
            if (tau == ~0ull) break;  // fewer middle slots than E
            // keys are distinct (they hold the position), so one thread owns the minimum
            if (LK && best == tau) s_ev[r] = best_j;
            ++found;
        }
        thr = tau;
        shift = 0;
        if (LK) {
            // Holes: evicted slots below the budget; movers: kept slots at or
            // above it; the k-th mover fills the k-th hole, both in slot order
            // (at most kSmallE of each, so one thread pairs them).
            __syncthreads();
            if (tid == 0) {
                int holes[kSmallE], nh = 0;
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
                s_nm = nm;
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
    int32_t* src = LK ? s_src : ws_src + static_cast<size_t>(l) * cap;
    int32_t* dst = LK ? s_dst : ws_dst + static_cast<size_t>(l) * cap;
    int n_moves = 0;
    if (LK && E > 0 && E <= kSmallE) {
        n_moves = s_nm;  // paired above
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
        if (!LK && tid == 0) ws_n[l] = n_moves;
        __syncthreads();
    }

    for (int r = tid; r < n_moves; r += kSel) {
        const int s = src[r], d = dst[r];
        A[d] = A[s];
        P[d] = P[s];
    }
    if (LK || inline_kv) {
        const int total = n_moves * Hkv * 2 * CH;
        for (int i = tid; i < total; i += kSel) {
            const int c = i % CH;
            int t = i / CH;
            const int which = t & 1;
            t >>= 1;
            const int h = t % Hkv, r = t / Hkv;
            T* base = (which ? v_cache : k_cache) + (static_cast<size_t>(l) * Hkv + h) * cap * D + c * PER;
            *reinterpret_cast<uint4*>(base + static_cast<size_t>(dst[r]) * D) =
                *reinterpret_cast<const uint4*>(base + static_cast<size_t>(src[r]) * D);
        }
    }

    if (kept_pos_out) {
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
        int32_t* outp = kept_pos_out + static_cast<size_t>(l) * budget;
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

template <int DT, int D>
__global__ __launch_bounds__(256) void compact_kernel(typename vz::Elem<DT>::T* __restrict__ k_cache,
                                                      typename vz::Elem<DT>::T* __restrict__ v_cache,
                                                      const int32_t* __restrict__ ws_n,
                                                      const int32_t* __restrict__ ws_src,
                                                      const int32_t* __restrict__ ws_dst, int32_t Hkv, int32_t cap) {
    using T = typename vz::Elem<DT>::T;
    constexpr int PER = vz::Elem<DT>::kPer16B;
    constexpr int CH = D / PER;
    const int l = blockIdx.y;
    const int n = ws_n[l];
    const int32_t* src = ws_src + static_cast<size_t>(l) * cap;
    const int32_t* dst = ws_dst + static_cast<size_t>(l) * cap;
    const int64_t total = static_cast<int64_t>(n) * Hkv * 2 * CH;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < total;
         i += static_cast<int64_t>(gridDim.x) * 256) {
        const int c = static_cast<int>(i % CH);
        int64_t t = i / CH;
        const int which = static_cast<int>(t & 1);
        t >>= 1;
        const int h = static_cast<int>(t % Hkv);
        const int r = static_cast<int>(t / Hkv);
        T* base = (which ? v_cache : k_cache) + (static_cast<size_t>(l) * Hkv + h) * cap * D + c * PER;
        *reinterpret_cast<uint4*>(base + static_cast<size_t>(dst[r]) * D) =
            *reinterpret_cast<const uint4*>(base + static_cast<size_t>(src[r]) * D);
    }
}

template <int DT, int D>
hipError_t launch(const VzEvictArgs& a, hipStream_t stream) {
    using T = typename vz::Elem<DT>::T;
    constexpr int CH = D / vz::Elem<DT>::kPer16B;
    const int E = a.len > a.budget ? a.len - a.budget : 0;
    if (E == 0 && a.kept_pos_out == nullptr) return hipSuccess;
    int32_t* ws_n = static_cast<int32_t*>(a.ws);
    int32_t* ws_src = ws_n + 64 * ((a.L + 63) / 64);
    int32_t* ws_dst = ws_src + static_cast<size_t>(a.L) * a.cap;
    const int M = a.n_recent < 0 ? a.budget / 5 : a.n_recent;
    const int inline_kv = E <= kInlineRows ? 1 : 0;
    if (inline_kv && a.len <= kLdsSlots)
        hipLaunchKernelGGL((select_kernel<DT, D, true>), dim3(a.L), dim3(kSel), 0, stream, static_cast<T*>(a.k_cache),
                           static_cast<T*>(a.v_cache), a.score, a.pos, a.len, a.budget, a.n_sink, M, a.next_pos,
                           a.kept_pos_out, a.Hkv, a.cap, ws_n, ws_src, ws_dst, inline_kv);
    else
        hipLaunchKernelGGL((select_kernel<DT, D, false>), dim3(a.L), dim3(kSel), 0, stream,
                           static_cast<T*>(a.k_cache), static_cast<T*>(a.v_cache), a.score, a.pos, a.len, a.budget,
                           a.n_sink, M, a.next_pos, a.kept_pos_out, a.Hkv, a.cap, ws_n, ws_src, ws_dst, inline_kv);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || inline_kv) return e;
    const int64_t chunks = static_cast<int64_t>(E) * a.Hkv * 2 * CH;
    const int gx = static_cast<int>(std::min<int64_t>((chunks + 255) / 256, 2048));
    hipLaunchKernelGGL((compact_kernel<DT, D>), dim3(gx, a.L), dim3(256), 0, stream, static_cast<T*>(a.k_cache),
                       static_cast<T*>(a.v_cache), ws_n, ws_src, ws_dst, a.Hkv, a.cap);
    return hipGetLastError();
}

}  // namespace

size_t vz_evict_ws_bytes(int32_t L, int32_t /*Hkv*/, int32_t /*d*/, int32_t cap) {
    return (static_cast<size_t>(64) * ((L + 63) / 64) + 2 * static_cast<size_t>(L) * cap) * sizeof(int32_t);
}

hipError_t vz_launch_evict(const VzEvictArgs& a, hipStream_t stream) {
    if (a.dtype == VZ_BF16 && a.d == 128) return launch<VZ_BF16, 128>(a, stream);
    if (a.dtype == VZ_BF16 && a.d == 64) return launch<VZ_BF16, 64>(a, stream);
    if (a.dtype == VZ_F32 && a.d == 128) return launch<VZ_F32, 128>(a, stream);
    if (a.dtype == VZ_F32 && a.d == 64) return launch<VZ_F32, 64>(a, stream);
    return hipErrorInvalidValue;
}
