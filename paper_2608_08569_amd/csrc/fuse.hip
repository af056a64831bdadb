// Stage-1 semantic-anchored fusion (Sec. 3.2.1, Eq. 4 group means plus the
// additive anchor, Eq. 5 order) as a segmented mean over K/V rows.
// Head sizes 64 and 128 (K/V-space fusion) use the lane-group kernel below;
// wider rows -- the embedding-space form, one "head" of width d_model -- use
// a kernel with one block per span that sweeps the row in 16-byte columns.
// Either kernel fuses K and V, or K alone when no V is given.
//
// Work split: a "lane group" of D/ (16 bytes / element size) lanes owns one
// (layer, KV head, K-or-V, span); each lane owns 16 contiguous bytes of the
// row, so a group reads whole rows with 16-byte loads and a wave streams
// 64 * 16 = 1 KB per load instruction.  Rows of a span are contiguous in HBM;
// the loop keeps four rows in flight per lane.  Accumulation is float32 in row
// order; the mean is an IEEE division by the span length, so a length-1 span
// reproduces its row bit for bit.
#include "vz_internal.h"

namespace {

struct FuseArgs {
    const void* k_in;
    const void* v_in;
    const int32_t* off;
    const void* ak;
    const void* av;
    void* k_out;
    void* v_out;
    float* score_out;
    int32_t* pos_out;
    int32_t H;
    int32_t kinds;              // 2: K and V, 1: K only
    int32_t d;                  // row length (the wide-row kernel)
    int32_t T_in, n_spans;      // single sequence
    int64_t in_plane, out_plane;  // rows per (layer, head) plane of the input and of the output
    int32_t blocks_per_seq;     // ragged: span blocks per sequence in grid x
    // ragged batch (n_seqs > 0): sequence s reads input rows in_base[s] ..
    // + T_in[s] and offsets off[off_base[s] .. + n_spans[s]], writes output
    // slots base[s] .. + n_spans[s] (cap[s] slots are its own)
    int32_t n_seqs;
    const int64_t* in_base;
    const int32_t* T_in_s;
    const int64_t* off_base;
    const int32_t* n_spans_s;
    const int64_t* base;
    const int32_t* cap;
    int32_t* status;
    int64_t total_off;
    int32_t max_spans;
};

// Status of sequence s of a ragged fusion (VZ_OK when it can be served,
// VZ_IDLE for an idle slot).
__device__ int ragged_fuse_status(const FuseArgs& a, int s) {
    const int64_t ib = a.in_base[s], ob = a.off_base[s], b = a.base[s];
    const int T = a.T_in_s[s], n = a.n_spans_s[s], c = a.cap[s];
    if (c == 0) return VZ_IDLE;
    if (T < 0 || n < 0 || c < 1 || ib < 0 || ib > a.in_plane - T || ob < 0 || ob > a.total_off - n - 1 || b < 0 ||
        b > a.out_plane - c)
        return VZ_ERR_INVALID;
    if (n > T) return VZ_ERR_SHAPE;
    if (n > c || n > a.max_spans) return VZ_ERR_CAPACITY;
    return VZ_OK;
}

template <int DT, int D, bool RAG>
__global__ __launch_bounds__(256) void fuse_spans_kernel(const FuseArgs a) {
    using E = vz::Elem<DT>;
    using T = typename E::T;
    constexpr int PER = E::kPer16B;      // elements per 16-byte vector
    constexpr int LANES = D / PER;       // lanes per span row
    constexpr int SPB = 256 / LANES;     // spans per block

    const int sub = threadIdx.x / LANES;
    const int lane = threadIdx.x % LANES;
    const int which = blockIdx.y % a.kinds;  // 0: K, 1: V
    const int h = blockIdx.y / a.kinds;
    const int l = blockIdx.z;
    int bx = blockIdx.x, T_in = a.T_in, n_spans = a.n_spans;
    int64_t in_row = 0, out_row = 0;  // first row of the sequence in its planes
    const int32_t* off = a.off;
    if constexpr (RAG) {
        const int s = blockIdx.x / a.blocks_per_seq;
        bx = blockIdx.x - s * a.blocks_per_seq;
        const int st = ragged_fuse_status(a, s);
        if (a.status && bx == 0 && blockIdx.y == 0 && l == 0 && threadIdx.x == 0) a.status[s] = st;
        if (st != VZ_OK) return;
        T_in = a.T_in_s[s];
        n_spans = a.n_spans_s[s];
        in_row = a.in_base[s];
        out_row = a.base[s];
        off = a.off + a.off_base[s];
    }
    const int64_t j = static_cast<int64_t>(bx) * SPB + sub;
    if (j >= n_spans) return;

    int32_t b = off[j], e = off[j + 1];
    b = b < 0 ? 0 : (b > T_in ? T_in : b);
    e = e < b ? b : (e > T_in ? T_in : e);

    const T* src = static_cast<const T*>(which ? a.v_in : a.k_in) +
                   ((static_cast<size_t>(l) * a.H + h) * static_cast<size_t>(a.in_plane) + in_row) * D + lane * PER;
    float acc[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) acc[i] = 0.f;

    int32_t r = b;
    for (; r + 4 <= e; r += 4) {
        uint4 x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            x[u] = *reinterpret_cast<const uint4*>(src + static_cast<size_t>(r + u) * D);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            float f[PER];
            vz::unpack16<DT>(x[u], f);
#pragma unroll
            for (int i = 0; i < PER; ++i) acc[i] += f[i];
        }
    }
    for (; r < e; ++r) {
        uint4 x = *reinterpret_cast<const uint4*>(src + static_cast<size_t>(r) * D);
        float f[PER];
        vz::unpack16<DT>(x, f);
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] += f[i];
    }
    const float cnt = static_cast<float>(e - b);
#pragma unroll
    for (int i = 0; i < PER; ++i) acc[i] = (e > b) ? acc[i] / cnt : 0.f;

    const T* anchor = static_cast<const T*>(which ? a.av : a.ak);
    const size_t orow = (static_cast<size_t>(l) * a.H + h) * static_cast<size_t>(a.out_plane) + out_row + j;
    if (anchor) {
        // single sequence: [L][H][n_spans][d]; ragged: laid out like the output
        const size_t arow = RAG ? orow : (static_cast<size_t>(l) * a.H + h) * static_cast<size_t>(n_spans) + j;
        uint4 x = *reinterpret_cast<const uint4*>(anchor + arow * D + lane * PER);
        float f[PER];
        vz::unpack16<DT>(x, f);
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] += f[i];
    }
    T* dst = static_cast<T*>(which ? a.v_out : a.k_out) + orow * D + lane * PER;
    *reinterpret_cast<uint4*>(dst) = vz::pack16<DT>(acc);

    if (which == 0 && h == 0 && lane == 0) {
        const size_t prow = static_cast<size_t>(l) * a.out_plane + out_row + j;
        a.pos_out[prow] = static_cast<int32_t>(j);
        a.score_out[prow] = 0.f;
    }
}

// Wide rows (d a multiple of one 16-byte vector, other than 64 and 128): one
// block of WIDE_THREADS threads per (span, K-or-V, head, layer); thread t
// owns the 16-byte columns t, t + WIDE_THREADS, ... of the row and sums them
// over the span's rows in row order (4 rows in flight), as the lane-group
// kernel does, so the arithmetic is the same.
constexpr int WIDE_THREADS = 256;
template <int DT, bool RAG>
__global__ __launch_bounds__(WIDE_THREADS) void fuse_wide_kernel(const FuseArgs a) {
    using E = vz::Elem<DT>;
    using T = typename E::T;
    constexpr int PER = E::kPer16B;
    const int nv = a.d / PER;  // 16-byte columns per row
    const int which = blockIdx.y % a.kinds;
    const int h = blockIdx.y / a.kinds;
    const int l = blockIdx.z;
    int64_t j = blockIdx.x;
    int T_in = a.T_in, n_spans = a.n_spans;
    int64_t in_row = 0, out_row = 0;
    const int32_t* off = a.off;
    if constexpr (RAG) {
        const int s = static_cast<int>(blockIdx.x / a.blocks_per_seq);
        j = blockIdx.x - static_cast<int64_t>(s) * a.blocks_per_seq;
        const int st = ragged_fuse_status(a, s);
        if (a.status && j == 0 && blockIdx.y == 0 && l == 0 && threadIdx.x == 0) a.status[s] = st;
        if (st != VZ_OK) return;
        T_in = a.T_in_s[s];
        n_spans = a.n_spans_s[s];
        in_row = a.in_base[s];
        out_row = a.base[s];
        off = a.off + a.off_base[s];
    }
    if (j >= n_spans) return;
    int32_t b = off[j], e = off[j + 1];
    b = b < 0 ? 0 : (b > T_in ? T_in : b);
    e = e < b ? b : (e > T_in ? T_in : e);
    const float cnt = static_cast<float>(e - b);
    const T* src = static_cast<const T*>(which ? a.v_in : a.k_in) +
                   ((static_cast<size_t>(l) * a.H + h) * static_cast<size_t>(a.in_plane) + in_row) * a.d;
    const T* anchor = static_cast<const T*>(which ? a.av : a.ak);
    const size_t orow = (static_cast<size_t>(l) * a.H + h) * static_cast<size_t>(a.out_plane) + out_row + j;
    const size_t arow = RAG ? orow : (static_cast<size_t>(l) * a.H + h) * static_cast<size_t>(n_spans) + j;
    T* dst = static_cast<T*>(which ? a.v_out : a.k_out) + orow * a.d;
    for (int c = threadIdx.x; c < nv; c += WIDE_THREADS) {
        const T* col = src + c * PER;
        float acc[PER];
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] = 0.f;
        int32_t r = b;
        for (; r + 4 <= e; r += 4) {
            uint4 x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) x[u] = *reinterpret_cast<const uint4*>(col + static_cast<size_t>(r + u) * a.d);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                float f[PER];
                vz::unpack16<DT>(x[u], f);
#pragma unroll
                for (int i = 0; i < PER; ++i) acc[i] += f[i];
            }
        }
        for (; r < e; ++r) {
            const uint4 x = *reinterpret_cast<const uint4*>(col + static_cast<size_t>(r) * a.d);
            float f[PER];
            vz::unpack16<DT>(x, f);
#pragma unroll
            for (int i = 0; i < PER; ++i) acc[i] += f[i];
        }
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] = (e > b) ? acc[i] / cnt : 0.f;
        if (anchor) {
            const uint4 x = *reinterpret_cast<const uint4*>(anchor + arow * a.d + c * PER);
            float f[PER];
            vz::unpack16<DT>(x, f);
#pragma unroll
            for (int i = 0; i < PER; ++i) acc[i] += f[i];
        }
        *reinterpret_cast<uint4*>(dst + c * PER) = vz::pack16<DT>(acc);
    }
    if (which == 0 && h == 0 && threadIdx.x == 0) {
        const size_t prow = static_cast<size_t>(l) * a.out_plane + out_row + j;
        a.pos_out[prow] = static_cast<int32_t>(j);
        a.score_out[prow] = 0.f;
    }
}

template <int DT>
hipError_t launch_wide(const FuseArgs& a, int32_t L, hipStream_t stream) {
    if (a.n_seqs > 0) {
        FuseArgs r = a;
        r.blocks_per_seq = a.max_spans > 0 ? a.max_spans : 1;  // still report every sequence's status
        dim3 grid(static_cast<unsigned>(static_cast<int64_t>(r.blocks_per_seq) * a.n_seqs), a.kinds * a.H, L);
        hipLaunchKernelGGL((fuse_wide_kernel<DT, true>), grid, dim3(WIDE_THREADS), 0, stream, r);
        return hipGetLastError();
    }
    if (a.n_spans == 0) return hipSuccess;
    dim3 grid(a.n_spans, a.kinds * a.H, L);
    hipLaunchKernelGGL((fuse_wide_kernel<DT, false>), grid, dim3(WIDE_THREADS), 0, stream, a);
    return hipGetLastError();
}

template <int DT, int D>
hipError_t launch(const FuseArgs& a, int32_t L, hipStream_t stream) {
    constexpr int SPB = 256 / (D / vz::Elem<DT>::kPer16B);
    if (a.n_seqs > 0) {
        FuseArgs r = a;
        r.blocks_per_seq = (a.max_spans + SPB - 1) / SPB;
        if (r.blocks_per_seq == 0) r.blocks_per_seq = 1;  // still report every sequence's status
        dim3 grid(static_cast<unsigned>(static_cast<int64_t>(r.blocks_per_seq) * a.n_seqs), a.kinds * a.H, L);
        hipLaunchKernelGGL((fuse_spans_kernel<DT, D, true>), grid, dim3(256), 0, stream, r);
        return hipGetLastError();
    }
    if (a.n_spans == 0) return hipSuccess;
    dim3 grid((a.n_spans + SPB - 1) / SPB, a.kinds * a.H, L);
    hipLaunchKernelGGL((fuse_spans_kernel<DT, D, false>), grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t dispatch(FuseArgs a, int32_t L, int32_t d, int32_t dtype, hipStream_t stream) {
    a.kinds = a.v_in ? 2 : 1;
    a.d = d;
    if (dtype == VZ_BF16 && d == 128) return launch<VZ_BF16, 128>(a, L, stream);
    if (dtype == VZ_BF16 && d == 64) return launch<VZ_BF16, 64>(a, L, stream);
    if (dtype == VZ_F32 && d == 128) return launch<VZ_F32, 128>(a, L, stream);
    if (dtype == VZ_F32 && d == 64) return launch<VZ_F32, 64>(a, L, stream);
    if (dtype == VZ_BF16 && d % vz::Elem<VZ_BF16>::kPer16B == 0) return launch_wide<VZ_BF16>(a, L, stream);
    if (dtype == VZ_F32 && d % vz::Elem<VZ_F32>::kPer16B == 0) return launch_wide<VZ_F32>(a, L, stream);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t vz_launch_fuse(const void* k_in, const void* v_in, int32_t T_in, const int32_t* off,
                          int32_t n_spans, const void* ak, const void* av, void* k_out, void* v_out,
                          float* score_out, int32_t* pos_out, int32_t L, int32_t H, int32_t d,
                          int32_t cap_out, int32_t dtype, hipStream_t stream) {
    FuseArgs a{};
    a.k_in = k_in;
    a.v_in = v_in;
    a.off = off;
    a.ak = ak;
    a.av = av;
    a.k_out = k_out;
    a.v_out = v_out;
    a.score_out = score_out;
    a.pos_out = pos_out;
    a.H = H;
    a.T_in = T_in;
    a.n_spans = n_spans;
    a.in_plane = T_in;
    a.out_plane = cap_out;
    return dispatch(a, L, d, dtype, stream);
}

hipError_t vz_launch_fuse_ragged(const VzFuseRaggedArgs& g, hipStream_t stream) {
    FuseArgs a{};
    a.k_in = g.k_in;
    a.v_in = g.v_in;
    a.off = g.span_off;
    a.ak = g.anchor_k;
    a.av = g.anchor_v;
    a.k_out = g.k_out;
    a.v_out = g.v_out;
    a.score_out = g.score_out;
    a.pos_out = g.pos_out;
    a.H = g.Hkv;
    a.in_plane = g.total_in;
    a.out_plane = g.total;
    a.n_seqs = g.n_seqs;
    a.in_base = g.in_base;
    a.T_in_s = g.T_in;
    a.off_base = g.off_base;
    a.n_spans_s = g.n_spans;
    a.base = g.seq_base;
    a.cap = g.cap;
    a.status = g.status;
    a.total_off = g.total_off;
    a.max_spans = g.max_spans;
    return dispatch(a, g.L, g.d, g.dtype, stream);
}
