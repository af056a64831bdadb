// Stage-1 semantic-anchored fusion (Sec. 3.2.1, Eq. 4 group means plus the
// additive anchor, Eq. 5 order) as a segmented mean over K/V rows.
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

template <int DT, int D>
__global__ __launch_bounds__(256) void fuse_spans_kernel(
    const typename vz::Elem<DT>::T* __restrict__ k_in, const typename vz::Elem<DT>::T* __restrict__ v_in,
    int32_t T_in, const int32_t* __restrict__ off, int32_t n_spans,
    const typename vz::Elem<DT>::T* __restrict__ ak, const typename vz::Elem<DT>::T* __restrict__ av,
    typename vz::Elem<DT>::T* __restrict__ k_out, typename vz::Elem<DT>::T* __restrict__ v_out,
    float* __restrict__ score_out, int32_t* __restrict__ pos_out, int32_t H, int32_t cap_out) {
    using E = vz::Elem<DT>;
    using T = typename E::T;
    constexpr int PER = E::kPer16B;      // elements per 16-byte vector
    constexpr int LANES = D / PER;       // lanes per span row
    constexpr int SPB = 256 / LANES;     // spans per block

    const int sub = threadIdx.x / LANES;
    const int lane = threadIdx.x % LANES;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * SPB + sub;
    if (j >= n_spans) return;
    const int which = blockIdx.y & 1;    // 0: K, 1: V
    const int h = blockIdx.y >> 1;
    const int l = blockIdx.z;

    int32_t b = off[j], e = off[j + 1];
    b = b < 0 ? 0 : (b > T_in ? T_in : b);
    e = e < b ? b : (e > T_in ? T_in : e);

    const T* src = (which ? v_in : k_in) + (static_cast<size_t>(l) * H + h) * static_cast<size_t>(T_in) * D +
                   lane * PER;
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

    const T* anchor = which ? av : ak;
    const size_t orow = (static_cast<size_t>(l) * H + h) * static_cast<size_t>(cap_out) + j;
    if (anchor) {
        const size_t arow = (static_cast<size_t>(l) * H + h) * static_cast<size_t>(n_spans) + j;
        uint4 x = *reinterpret_cast<const uint4*>(anchor + arow * D + lane * PER);
        float f[PER];
        vz::unpack16<DT>(x, f);
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] += f[i];
    }
    T* dst = (which ? v_out : k_out) + orow * D + lane * PER;
    *reinterpret_cast<uint4*>(dst) = vz::pack16<DT>(acc);

    if (which == 0 && h == 0 && lane == 0) {
        pos_out[static_cast<size_t>(l) * cap_out + j] = static_cast<int32_t>(j);
        score_out[static_cast<size_t>(l) * cap_out + j] = 0.f;
    }
}

template <int DT, int D>
hipError_t launch(const void* k_in, const void* v_in, int32_t T_in, const int32_t* off, int32_t n_spans,
                  const void* ak, const void* av, void* k_out, void* v_out, float* score_out,
                  int32_t* pos_out, int32_t L, int32_t H, int32_t cap_out, hipStream_t stream) {
    using T = typename vz::Elem<DT>::T;
    constexpr int SPB = 256 / (D / vz::Elem<DT>::kPer16B);
    if (n_spans == 0) return hipSuccess;
    dim3 grid((n_spans + SPB - 1) / SPB, 2 * H, L);
    hipLaunchKernelGGL((fuse_spans_kernel<DT, D>), grid, dim3(256), 0, stream,
                       static_cast<const T*>(k_in), static_cast<const T*>(v_in), T_in, off, n_spans,
                       static_cast<const T*>(ak), static_cast<const T*>(av), static_cast<T*>(k_out),
                       static_cast<T*>(v_out), score_out, pos_out, H, cap_out);
    return hipGetLastError();
}

}  // namespace

hipError_t vz_launch_fuse(const void* k_in, const void* v_in, int32_t T_in, const int32_t* off,
                          int32_t n_spans, const void* ak, const void* av, void* k_out, void* v_out,
                          float* score_out, int32_t* pos_out, int32_t L, int32_t H, int32_t d,
                          int32_t cap_out, int32_t dtype, hipStream_t stream) {
    if (dtype == VZ_BF16 && d == 128)
        return launch<VZ_BF16, 128>(k_in, v_in, T_in, off, n_spans, ak, av, k_out, v_out, score_out,
                                    pos_out, L, H, cap_out, stream);
    if (dtype == VZ_BF16 && d == 64)
        return launch<VZ_BF16, 64>(k_in, v_in, T_in, off, n_spans, ak, av, k_out, v_out, score_out,
                                   pos_out, L, H, cap_out, stream);
    if (dtype == VZ_F32 && d == 128)
        return launch<VZ_F32, 128>(k_in, v_in, T_in, off, n_spans, ak, av, k_out, v_out, score_out,
                                   pos_out, L, H, cap_out, stream);
    if (dtype == VZ_F32 && d == 64)
        return launch<VZ_F32, 64>(k_in, v_in, T_in, off, n_spans, ak, av, k_out, v_out, score_out,
                                  pos_out, L, H, cap_out, stream);
    return hipErrorInvalidValue;
}
