// Stage-2 eviction (Sec. 3.2.2, Eq. 7-9) with in-place hole-fill compaction:
// one 1024-thread block per layer (and sequence) runs the selection of
// select.h; layers with many moved rows finish their K/V moves in a grid-wide
// copy kernel.  When the layer has at most 16384 slots and at most 256 of them
// move (the steady state of one eviction per step, and most first evictions),
// the keys are computed once into LDS with one coalesced pass over score and
// pos, and the selection, the classification and the move lists all stay in
// LDS: the only other global round trip is the moved rows themselves.
#include <algorithm>
#include <type_traits>

#include "select.h"

namespace {

using namespace vz_sel;

constexpr int kSel = 1024;
constexpr int kLdsSlots = 16384;    // slots whose keys fit in LDS
static_assert(kLdsSlots % (2 * kSel) == 0, "one load round of the LDS keys");

template <bool LK>
using SelSh = SelShared<kSel, LK ? kLdsSlots : 0>;

// Single sequence: one block per layer.
template <int DT, int D, bool LK>
__global__ __launch_bounds__(kSel) void select_kernel(const VzEvictArgs a, int32_t M, int32_t* __restrict__ ws_n,
                                                      int32_t* __restrict__ ws_src, int32_t* __restrict__ ws_dst,
                                                      int inline_kv) {
    using T = typename vz::Elem<DT>::T;
    __shared__ SelSh<LK> sh;
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
    select_body<kSel, DT, D, LK>(job, sh);
}

// Status of sequence s for an eviction (VZ_OK when it can be served, VZ_IDLE
// for an idle slot).
__device__ int ragged_evict_status(const VzRagged& r, int s, int n_sink, int n_recent, bool kept) {
    const int64_t b = r.base[s];
    const int c = r.cap[s], n = r.len[s], B = r.budget[s], p = r.next_pos[s];
    if (c == 0) return VZ_IDLE;
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
    __shared__ SelSh<true> sh;
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
        select_body<kSel, DT, D, true>(job, sh);
    else
        select_body<kSel, DT, D, false>(job, sh);
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

