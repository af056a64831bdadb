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

// Arguments shared by the three launches (see the fused path: a
// single-sequence call has rag.n == 0).
struct GenericArgs {
    const void* q;
    const void* k_new;
    const void* v_new;
    void* k_cache;
    void* v_cache;
    int32_t* pos;
    float* score;
    void* out;
    float* S;    // logits [L][Hq][plane]
    float* ml;   // [seqs][L][Hq][2] max and sum of exp per head
    int32_t len, next_pos;  // single sequence
    int32_t n_blocks;       // key blocks per layer (grid extent)
    int32_t Hq, Hkv, L;
    int64_t plane;
    float scale, gamma;
    VzRagged rag;
};

__device__ __forceinline__ int ragged_blocks(const VzRagged& r, int s) {
    return vz::ragged_decode_status(r, s) == VZ_OK ? (r.len[s] + kThreads) / kThreads : 0;
}

struct SeqKeys {
    int s, len, next_pos;
    int64_t base;
};

// Key block f of a layer: false when it holds no work; c = block inside the sequence.
template <bool RAG>
__device__ __forceinline__ bool resolve_block(const GenericArgs& a, int f, SeqKeys& it, int& c) {
    if constexpr (RAG) {
        int first = 0, nb = 0;
        const int s = vz::ragged_locate(f, a.rag.n, a.n_blocks, [&](int t) { return ragged_blocks(a.rag, t); },
                                        first, nb);
        if (s < 0 || first + nb > a.n_blocks) return false;
        it.s = s;
        it.len = a.rag.len[s];
        it.next_pos = a.rag.next_pos[s];
        it.base = a.rag.base[s];
        c = f - first;
    } else {
        it.s = 0;
        it.len = a.len;
        it.next_pos = a.next_pos;
        it.base = 0;
        c = f;
    }
    return true;
}

template <int DT, int D, bool RAG>
__global__ __launch_bounds__(kThreads) void logits_kernel(const GenericArgs a) {
    using E = vz::Elem<DT>;
    using T = typename E::T;
    constexpr int PER = E::kPer16B;
    __shared__ float qs[16 * D];
    const int l = blockIdx.y;
    SeqKeys it;
    int c;
    if (!resolve_block<RAG>(a, blockIdx.x, it, c)) return;
    const int len = it.len;
    const int T_keys = len + 1;
    const int j = c * kThreads + threadIdx.x;
    const int Hq = a.Hq, Hkv = a.Hkv;
    const int G = Hq / Hkv;
    const size_t row_sl = static_cast<size_t>(it.s) * a.L + l;
    const T* q = static_cast<const T*>(a.q);
    const T* k_new = static_cast<const T*>(a.k_new);
    const T* v_new = static_cast<const T*>(a.v_new);
    T* k_cache = static_cast<T*>(a.k_cache);
    T* v_cache = static_cast<T*>(a.v_cache);

    for (int g = 0; g < Hkv; ++g) {
        __syncthreads();
        for (int i = threadIdx.x; i < G * D; i += kThreads)
            qs[i] = E::load(q, (row_sl * Hq + static_cast<size_t>(g) * G) * D + i);
        __syncthreads();
        if (j < T_keys) {
            const T* krow = (j < len) ? k_cache + ((static_cast<size_t>(l) * Hkv + g) * a.plane + it.base + j) * D
                                      : k_new + (row_sl * Hkv + g) * D;
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
                if (hh < G) a.S[(static_cast<size_t>(l) * Hq + g * G + hh) * a.plane + it.base + j] = acc[hh] * a.scale;
        }
    }
    if (j == len) {  // Eq. (1): append the new row to every KV head of this layer
        for (int g = 0; g < Hkv; ++g) {
            const size_t src = (row_sl * Hkv + g) * D;
            const size_t dst = ((static_cast<size_t>(l) * Hkv + g) * a.plane + it.base + len) * D;
            for (int c0 = 0; c0 < D; c0 += PER) {
                *reinterpret_cast<uint4*>(k_cache + dst + c0) = *reinterpret_cast<const uint4*>(k_new + src + c0);
                *reinterpret_cast<uint4*>(v_cache + dst + c0) = *reinterpret_cast<const uint4*>(v_new + src + c0);
            }
        }
        a.pos[static_cast<size_t>(l) * a.plane + it.base + len] = it.next_pos;
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

// One block per (head, layer, sequence); in a ragged call also stores the
// sequence's status.
template <int DT, int D, bool RAG>
__global__ __launch_bounds__(kThreads) void combine_kernel(const GenericArgs a) {
    using E = vz::Elem<DT>;
    constexpr int JL = kThreads / D;
    __shared__ float red[kThreads / vz::kWave];
    __shared__ float part[kThreads];
    const int h = blockIdx.x, l = blockIdx.y;
    int s = 0, len = a.len;
    int64_t base = 0;
    if constexpr (RAG) {
        s = blockIdx.z;
        const int st = vz::ragged_decode_status(a.rag, s);
        int ok = st == VZ_OK;
        if (ok) {
            const int first = vz::ragged_first(s, a.n_blocks, [&](int t) { return ragged_blocks(a.rag, t); });
            ok = first >= 0 && first + ragged_blocks(a.rag, s) <= a.n_blocks;
        }
        if (a.rag.status && h == 0 && l == 0 && threadIdx.x == 0)
            a.rag.status[s] = ok ? VZ_OK : (st != VZ_OK ? st : VZ_ERR_CAPACITY);
        if (!ok) return;
        len = a.rag.len[s];
        base = a.rag.base[s];
    }
    const int Hq = a.Hq;
    const int T_keys = len + 1;
    const int g = h / (Hq / a.Hkv);
    const float* sv = a.S + (static_cast<size_t>(l) * Hq + h) * a.plane + base;
    const size_t row_sl = static_cast<size_t>(s) * a.L + l;

    float m = -INFINITY;
    for (int j = threadIdx.x; j < T_keys; j += kThreads) m = fmaxf(m, sv[j]);
    m = block_reduce(m, true, red);
    float z = 0.f;
    for (int j = threadIdx.x; j < T_keys; j += kThreads) z += expf(sv[j] - m);
    z = block_reduce(z, false, red);
    if (threadIdx.x == 0) {
        a.ml[(row_sl * Hq + h) * 2] = m;
        a.ml[(row_sl * Hq + h) * 2 + 1] = z;
    }
    const int c = threadIdx.x % D, jl = threadIdx.x / D;
    const typename E::T* V =
        static_cast<const typename E::T*>(a.v_cache) + ((static_cast<size_t>(l) * a.Hkv + g) * a.plane + base) * D;
    float acc = 0.f;
    for (int j = jl; j < T_keys; j += JL) acc += expf(sv[j] - m) * E::load(V, static_cast<size_t>(j) * D + c);
    part[threadIdx.x] = acc;
    __syncthreads();
    if (jl == 0) {
        float t = part[c];
        for (int i = 1; i < JL; ++i) t += part[i * D + c];
        static_cast<typename E::T*>(a.out)[(row_sl * Hq + h) * D + c] = E::from_f32(t / z);
    }
}

template <bool RAG>
__global__ __launch_bounds__(kThreads) void fold_kernel(const GenericArgs a) {
    __shared__ float mls[2 * 256];
    const int l = blockIdx.y;
    SeqKeys it;
    int c;
    if (!resolve_block<RAG>(a, blockIdx.x, it, c)) return;
    const int Hq = a.Hq;
    const size_t row_sl = static_cast<size_t>(it.s) * a.L + l;
    for (int i = threadIdx.x; i < 2 * Hq; i += kThreads) mls[i] = a.ml[row_sl * Hq * 2 + i];
    __syncthreads();
    const int len = it.len;
    const int j = c * kThreads + threadIdx.x;
    if (j > len) return;
    float* sc = a.score + static_cast<size_t>(l) * a.plane + it.base;
    float acc = (j < len) ? a.gamma * sc[j] : 0.f;
    for (int h = 0; h < Hq; ++h)
        acc += expf(a.S[(static_cast<size_t>(l) * Hq + h) * a.plane + it.base + j] - mls[2 * h]) / mls[2 * h + 1];
    sc[j] = acc;
}

int64_t key_blocks(int64_t plane, int32_t n_seqs) {
    return n_seqs > 0 ? (plane + kThreads - 1) / kThreads + n_seqs : (plane + kThreads - 1) / kThreads;
}

template <int DT, int D, bool RAG>
hipError_t launch(const VzDecodeArgs& v, hipStream_t stream) {
    GenericArgs a{};
    a.q = v.q;
    a.k_new = v.k_new;
    a.v_new = v.v_new;
    a.k_cache = v.k_cache;
    a.v_cache = v.v_cache;
    a.pos = v.pos;
    a.score = v.score;
    a.out = v.out;
    a.Hq = v.Hq;
    a.Hkv = v.Hkv;
    a.L = v.L;
    a.plane = RAG ? v.rag.total : v.cap;
    a.S = reinterpret_cast<float*>(static_cast<uint8_t*>(v.ws) + vz_decode_hdr_bytes(v.L));
    a.ml = a.S + static_cast<size_t>(v.L) * v.Hq * a.plane;
    a.scale = v.sm_scale > 0.f ? v.sm_scale : 1.0f / sqrtf(static_cast<float>(D));
    a.gamma = v.gamma;
    a.rag = v.rag;
    int seqs = 1;
    if (RAG) {
        a.n_blocks = static_cast<int32_t>(key_blocks(v.rag.total, v.rag.n));
        seqs = v.rag.n;
    } else {
        a.len = v.len;
        a.next_pos = v.next_pos;
        a.n_blocks = (v.len + kThreads) / kThreads;
    }
    dim3 gk(a.n_blocks, a.L);
    hipLaunchKernelGGL((logits_kernel<DT, D, RAG>), gk, dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((combine_kernel<DT, D, RAG>), dim3(a.Hq, a.L, seqs), dim3(kThreads), 0, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((fold_kernel<RAG>), gk, dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

template <int DT, int D>
hipError_t launch_any(const VzDecodeArgs& v, hipStream_t stream) {
    return v.rag.n > 0 ? launch<DT, D, true>(v, stream) : launch<DT, D, false>(v, stream);
}

}  // namespace

bool vz_decode_generic_ok(int64_t plane, int32_t n_seqs) {
    return key_blocks(plane, n_seqs) < (int64_t(1) << 31);  // grid x
}

size_t vz_decode_generic_ws_bytes(int32_t L, int32_t Hq, int64_t plane, int32_t n_seqs) {
    const int32_t seqs = n_seqs > 0 ? n_seqs : 1;
    return vz_decode_hdr_bytes(L) +
           (static_cast<size_t>(L) * Hq * plane + static_cast<size_t>(seqs) * L * Hq * 2) * sizeof(float);
}

hipError_t vz_launch_decode_generic(const VzDecodeArgs& a, hipStream_t stream) {
    if (a.dtype == VZ_BF16 && a.d == 128) return launch_any<VZ_BF16, 128>(a, stream);
    if (a.dtype == VZ_BF16 && a.d == 64) return launch_any<VZ_BF16, 64>(a, stream);
    if (a.dtype == VZ_F32 && a.d == 128) return launch_any<VZ_F32, 128>(a, stream);
    if (a.dtype == VZ_F32 && a.d == 64) return launch_any<VZ_F32, 64>(a, stream);
    return hipErrorInvalidValue;
}
