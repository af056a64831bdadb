// Decode step (Sec. 3.1 Eq. 1-2, Sec. 3.2.2 Eq. 6), general path: any group
// size up to 16, float32 or bfloat16, d in {64, 128}.  Three launches:
//
//   logits   one thread per key: s[l][h][j] = scale * q_h . K[g][j] for the
//            heads of every KV group (queries staged in LDS); the thread that
//            owns slot len appends k_new / v_new / next_pos first (it reads the
//            new key from k_new, so no other thread depends on that write);
//   combine  one block per (layer, head): max and sum of exp over the logits,
//            then o = sum_j exp(s_j - m) V[g][j] / sum with D channels x
//            (256 / D) key lanes;
//   fold     one thread per key: A[j] = gamma * A[j] + sum_h exp(s_hj - m_h) / l_h.
//
// The logits live in the workspace between launches.  This path is the one
// float32 caches use; bfloat16 caches with d = 128 take the fused MFMA path.
#include <math.h>

#include "vz_internal.h"

namespace {

constexpr int kThreads = 256;

template <int DT, int D>
__global__ __launch_bounds__(kThreads) void logits_kernel(
    const typename vz::Elem<DT>::T* __restrict__ q, const typename vz::Elem<DT>::T* __restrict__ k_new,
    const typename vz::Elem<DT>::T* __restrict__ v_new, typename vz::Elem<DT>::T* __restrict__ k_cache,
    typename vz::Elem<DT>::T* __restrict__ v_cache, int32_t* __restrict__ pos, float* __restrict__ S,
    int32_t len, int32_t next_pos, float scale, int32_t Hq, int32_t Hkv, int32_t cap) {
    using E = vz::Elem<DT>;
    using T = typename E::T;
    constexpr int PER = E::kPer16B;
    __shared__ float qs[16 * D];
    const int l = blockIdx.y;
    const int T_keys = len + 1;
    const int j = blockIdx.x * kThreads + threadIdx.x;
    const int G = Hq / Hkv;

    for (int g = 0; g < Hkv; ++g) {
        __syncthreads();
        for (int i = threadIdx.x; i < G * D; i += kThreads)
            qs[i] = E::load(q, (static_cast<size_t>(l) * Hq + static_cast<size_t>(g) * G) * D + i);
        __syncthreads();
        if (j < T_keys) {
            const T* krow = (j < len)
                                ? k_cache + ((static_cast<size_t>(l) * Hkv + g) * cap + j) * D
                                : k_new + (static_cast<size_t>(l) * Hkv + g) * D;
            float acc[16];
#pragma unroll
            for (int hh = 0; hh < 16; ++hh) acc[hh] = 0.f;
            for (int c0 = 0; c0 < D; c0 += PER) {
                float f[PER];
                vz::unpack16<DT>(*reinterpret_cast<const uint4*>(krow + c0), f);
#pragma unroll
                for (int hh = 0; hh < 16; ++hh) {
                    if (hh < G) {
#pragma unroll
                        for (int i = 0; i < PER; ++i) acc[hh] += qs[hh * D + c0 + i] * f[i];
                    }
                }
            }
#pragma unroll
            for (int hh = 0; hh < 16; ++hh)
                if (hh < G) S[(static_cast<size_t>(l) * Hq + g * G + hh) * cap + j] = acc[hh] * scale;
        }
    }
    if (j == len) {  // Eq. (1): append the new row to every KV head of this layer
        for (int g = 0; g < Hkv; ++g) {
            const size_t src = (static_cast<size_t>(l) * Hkv + g) * D;
            const size_t dst = ((static_cast<size_t>(l) * Hkv + g) * cap + len) * D;
            for (int c0 = 0; c0 < D; c0 += PER) {
                *reinterpret_cast<uint4*>(k_cache + dst + c0) = *reinterpret_cast<const uint4*>(k_new + src + c0);
                *reinterpret_cast<uint4*>(v_cache + dst + c0) = *reinterpret_cast<const uint4*>(v_new + src + c0);
            }
        }
        pos[static_cast<size_t>(l) * cap + len] = next_pos;
    }
}

__device__ float block_reduce(float v, bool is_max, float* red) {
    v = is_max ? vz::wave_max(v) : vz::wave_sum(v);
    const int w = threadIdx.x / vz::kWave;
    __syncthreads();
    if ((threadIdx.x % vz::kWave) == 0) red[w] = v;
    __syncthreads();
    float r = red[0];
    for (int i = 1; i < kThreads / vz::kWave; ++i) r = is_max ? fmaxf(r, red[i]) : r + red[i];
    return r;
}

template <int DT, int D>
__global__ __launch_bounds__(kThreads) void combine_kernel(
    const typename vz::Elem<DT>::T* __restrict__ v_cache, const float* __restrict__ S, float* __restrict__ ml,
    typename vz::Elem<DT>::T* __restrict__ out, int32_t len, int32_t Hq, int32_t Hkv, int32_t cap) {
    using E = vz::Elem<DT>;
    constexpr int JL = kThreads / D;
    __shared__ float red[kThreads / vz::kWave];
    __shared__ float part[kThreads];
    const int h = blockIdx.x, l = blockIdx.y;
    const int T_keys = len + 1;
    const int g = h / (Hq / Hkv);
    const float* s = S + (static_cast<size_t>(l) * Hq + h) * cap;

    float m = -INFINITY;
    for (int j = threadIdx.x; j < T_keys; j += kThreads) m = fmaxf(m, s[j]);
    m = block_reduce(m, true, red);
    float z = 0.f;
    for (int j = threadIdx.x; j < T_keys; j += kThreads) z += expf(s[j] - m);
    z = block_reduce(z, false, red);
    if (threadIdx.x == 0) {
        ml[(static_cast<size_t>(l) * Hq + h) * 2] = m;
        ml[(static_cast<size_t>(l) * Hq + h) * 2 + 1] = z;
    }
    const int c = threadIdx.x % D, jl = threadIdx.x / D;
    const typename E::T* V = v_cache + (static_cast<size_t>(l) * Hkv + g) * cap * D;
    float acc = 0.f;
    for (int j = jl; j < T_keys; j += JL) acc += expf(s[j] - m) * E::load(V, static_cast<size_t>(j) * D + c);
    part[threadIdx.x] = acc;
    __syncthreads();
    if (jl == 0) {
        float t = part[c];
        for (int i = 1; i < JL; ++i) t += part[i * D + c];
        out[(static_cast<size_t>(l) * Hq + h) * D + c] = E::from_f32(t / z);
    }
}

__global__ __launch_bounds__(kThreads) void fold_kernel(const float* __restrict__ S, const float* __restrict__ ml,
                                                        float* __restrict__ score, int32_t len, float gamma,
                                                        int32_t Hq, int32_t cap) {
    __shared__ float mls[2 * 256];
    const int l = blockIdx.y;
    for (int i = threadIdx.x; i < 2 * Hq; i += kThreads) mls[i] = ml[static_cast<size_t>(l) * Hq * 2 + i];
    __syncthreads();
    const int j = blockIdx.x * kThreads + threadIdx.x;
    if (j > len) return;
    float a = (j < len) ? gamma * score[static_cast<size_t>(l) * cap + j] : 0.f;
    for (int h = 0; h < Hq; ++h)
        a += expf(S[(static_cast<size_t>(l) * Hq + h) * cap + j] - mls[2 * h]) / mls[2 * h + 1];
    score[static_cast<size_t>(l) * cap + j] = a;
}

template <int DT, int D>
hipError_t launch(const VzDecodeArgs& a, hipStream_t stream) {
    using T = typename vz::Elem<DT>::T;
    float* S = reinterpret_cast<float*>(static_cast<uint8_t*>(a.ws) + vz_decode_hdr_bytes(a.L));
    float* ml = S + static_cast<size_t>(a.L) * a.Hq * a.cap;
    const float scale = a.sm_scale > 0.f ? a.sm_scale : 1.0f / sqrtf(static_cast<float>(D));
    const int T_keys = a.len + 1;
    dim3 gk((T_keys + kThreads - 1) / kThreads, a.L);
    hipLaunchKernelGGL((logits_kernel<DT, D>), gk, dim3(kThreads), 0, stream, static_cast<const T*>(a.q),
                       static_cast<const T*>(a.k_new), static_cast<const T*>(a.v_new), static_cast<T*>(a.k_cache),
                       static_cast<T*>(a.v_cache), a.pos, S, a.len, a.next_pos, scale, a.Hq, a.Hkv, a.cap);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((combine_kernel<DT, D>), dim3(a.Hq, a.L), dim3(kThreads), 0, stream,
                       static_cast<const T*>(a.v_cache), S, ml, static_cast<T*>(a.out), a.len, a.Hq, a.Hkv, a.cap);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fold_kernel, gk, dim3(kThreads), 0, stream, S, ml, a.score, a.len, a.gamma, a.Hq, a.cap);
    return hipGetLastError();
}

}  // namespace

size_t vz_decode_generic_ws_bytes(int32_t L, int32_t Hq, int32_t cap) {
    return vz_decode_hdr_bytes(L) + (static_cast<size_t>(L) * Hq * cap + static_cast<size_t>(L) * Hq * 2) * sizeof(float);
}

hipError_t vz_launch_decode_generic(const VzDecodeArgs& a, hipStream_t stream) {
    if (a.dtype == VZ_BF16 && a.d == 128) return launch<VZ_BF16, 128>(a, stream);
    if (a.dtype == VZ_BF16 && a.d == 64) return launch<VZ_BF16, 64>(a, stream);
    if (a.dtype == VZ_F32 && a.d == 128) return launch<VZ_F32, 128>(a, stream);
    if (a.dtype == VZ_F32 && a.d == 64) return launch<VZ_F32, 64>(a, stream);
    return hipErrorInvalidValue;
}
