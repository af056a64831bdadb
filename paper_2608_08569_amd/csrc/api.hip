// Host side of libvoxzip: argument validation, workspace sizing, status
// strings and dispatch to the kernel launchers.  Every check runs on the host
// before any HIP call, so invalid arguments never reach the GPU.
#include <math.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "vz_internal.h"

// Scratch memory of voxzip_decode_evict_noalloc: one array per GPU, held
// until the process ends.  In host code `scratch` names a host-side stand-in,
// not device memory: only the address hipGetSymbolAddress returns for the
// current device is ever used.
static __device__ __align__(256) uint8_t scratch[VZ_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fn, const char* what) {
    g_last_error = std::string(fn) + ": " + what;
    return status;
}

int hip_fail(const char* fn, hipError_t e) {
    g_last_error = std::string(fn) + ": " + hipGetErrorString(e);
    return VZ_ERR_HIP;
}

size_t elem_size(int32_t dtype) { return dtype == VZ_F32 ? 4 : 2; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const char* pa = static_cast<const char*>(a);
    const char* pb = static_cast<const char*>(b);
    return pa < pb + nb && pb < pa + na;
}

// Fusion also takes wide rows (the embedding-space form of Stage 1: one head of
// width d_model): any multiple of one 16-byte vector up to kFuseMaxD.
constexpr int32_t kFuseMaxD = 16384;

int check_common(const char* fn, int32_t L, int32_t Hkv, int32_t d, int32_t dtype, bool fusion = false) {
    if (L < 1 || Hkv < 1 || d < 1) return fail(VZ_ERR_SHAPE, fn, "sizes must be positive");
    if (dtype != VZ_F32 && dtype != VZ_BF16) return fail(VZ_ERR_UNSUPPORTED, fn, "dtype must be VZ_F32 or VZ_BF16");
    if (fusion) {
        const int32_t vec = dtype == VZ_F32 ? 4 : 8;  // elements per 16 bytes
        if (d != 64 && d != 128 && (d % vec != 0 || d > kFuseMaxD))
            return fail(VZ_ERR_UNSUPPORTED, fn, "row size must be 64, 128 or a multiple of 16 bytes up to 16384");
    } else if (d != 64 && d != 128) {
        return fail(VZ_ERR_UNSUPPORTED, fn, "head size must be 64 or 128");
    }
    if (L > 65535) return fail(VZ_ERR_UNSUPPORTED, fn, "more than 65535 layers");
    return VZ_OK;
}

// K and V, or K alone (v_in and v_out both NULL; then no anchor_v).
int check_fuse_pointers(const char* fn, const void* v_in, const void* v_out, const void* anchor_k,
                        const void* anchor_v) {
    if ((v_in == nullptr) != (v_out == nullptr))
        return fail(VZ_ERR_INVALID, fn, "v_in and v_out must both be given or both be NULL");
    if (v_in == nullptr) {
        if (anchor_v) return fail(VZ_ERR_INVALID, fn, "anchor_v given without v_in");
    } else if ((anchor_k == nullptr) != (anchor_v == nullptr)) {
        return fail(VZ_ERR_INVALID, fn, "anchor_k and anchor_v must both be given or both be NULL");
    }
    return VZ_OK;
}

int check_ragged(const char* fn, int32_t L, int32_t Hkv, int32_t d, int32_t dtype, int64_t total, int32_t n_seqs,
                 bool fusion = false) {
    int rc = check_common(fn, L, Hkv, d, dtype, fusion);
    if (rc) return rc;
    if (n_seqs < 1 || n_seqs > kRaggedMaxSeqs) return fail(VZ_ERR_SHAPE, fn, "n_seqs must be in [1, 32768]");
    if (total < 1 || total > kRaggedMaxTotal) return fail(VZ_ERR_SHAPE, fn, "total must be in [1, 2^26]");
    return VZ_OK;
}

// Arguments of a single-sequence decode step (shared by the decode entry
// points).
int check_decode(const char* fn, const void* q, const void* k_new, const void* v_new, const void* k_cache,
                 const void* v_cache, const float* score, const int32_t* pos, const void* out, int32_t len,
                 int32_t next_pos, float gamma, float sm_scale, int32_t n_layers, int32_t n_q_heads,
                 int32_t kv_heads, int32_t d, int32_t cap, int32_t dtype) {
    if (!q || !k_new || !v_new || !k_cache || !v_cache || !score || !pos || !out)
        return fail(VZ_ERR_INVALID, fn, "null pointer");
    int rc = check_common(fn, n_layers, kv_heads, d, dtype);
    if (rc) return rc;
    if (n_q_heads < 1 || n_q_heads % kv_heads != 0)
        return fail(VZ_ERR_SHAPE, fn, "n_q_heads must be a positive multiple of kv_heads");
    if (n_q_heads / kv_heads > 16) return fail(VZ_ERR_UNSUPPORTED, fn, "more than 16 query heads per KV head");
    if (n_q_heads > 256) return fail(VZ_ERR_UNSUPPORTED, fn, "more than 256 query heads");
    if (len < 0 || next_pos < 0) return fail(VZ_ERR_INVALID, fn, "negative len or next_pos");
    if (cap < 1 || len + 1 > cap) return fail(VZ_ERR_CAPACITY, fn, "no free slot for the new token");
    if (!(gamma >= 0.f && gamma <= 1.f)) return fail(VZ_ERR_INVALID, fn, "gamma must be in [0, 1]");
    if (!isfinite(sm_scale)) return fail(VZ_ERR_INVALID, fn, "sm_scale must be finite");
    return VZ_OK;
}

// Arguments of a single-sequence eviction of len slots; M receives the recent
// window.
int check_evict(const char* fn, int32_t len, int32_t budget, int32_t n_sink, int32_t n_recent, int32_t next_pos,
                const int32_t* kept_pos_out, int32_t cap, int32_t& M) {
    if (len < 0 || cap < 1) return fail(VZ_ERR_INVALID, fn, "negative len or empty cache");
    if (len > cap) return fail(VZ_ERR_CAPACITY, fn, "len exceeds cap");
    if (budget < 1 || n_sink < 0) return fail(VZ_ERR_INVALID, fn, "budget must be >= 1 and n_sink >= 0");
    M = n_recent < 0 ? budget / 5 : n_recent;
    if (static_cast<int64_t>(n_sink) + M > budget)
        return fail(VZ_ERR_INVALID, fn, "sink and recent windows exceed the budget");
    if (next_pos < len) return fail(VZ_ERR_INVALID, fn, "next_pos below len: positions cannot be distinct");
    if (kept_pos_out && next_pos > (1 << 18))
        return fail(VZ_ERR_UNSUPPORTED, fn, "kept_pos_out needs next_pos <= 262144");
    return VZ_OK;
}

// A workspace is usable when present, 16-byte aligned (its arrays are read
// and written with 16-byte accesses) and large enough.
bool ws_ok(const void* ws, size_t ws_bytes, size_t need) {
    return ws != nullptr && (reinterpret_cast<uintptr_t>(ws) & 15u) == 0 && ws_bytes >= need;
}

// A decode + evict workspace: the decode part, then the eviction part from
// the next 256-byte boundary.
size_t decode_evict_split(int32_t L, int32_t Hq, int32_t Hkv, int32_t d, int32_t cap) {
    return (vz_decode_ws_bytes(L, Hq, Hkv, d, cap, 0) + 255) / 256 * 256;
}

}  // namespace

extern "C" {

int voxzip_version(void) { return 100; }

const char* voxzip_last_error(void) { return g_last_error.c_str(); }

const char* voxzip_status_string(int status) {
    switch (status) {
        case VZ_OK: return "ok";
        case VZ_ERR_INVALID: return "invalid argument";
        case VZ_ERR_SHAPE: return "inconsistent shape";
        case VZ_ERR_CAPACITY: return "capacity exceeded";
        case VZ_ERR_UNSUPPORTED: return "unsupported configuration";
        case VZ_ERR_HIP: return "HIP error";
        case VZ_ERR_WORKSPACE: return "workspace too small";
        case VZ_IDLE: return "idle batch slot";
        default: return "unknown status";
    }
}

size_t voxzip_workspace_bytes(int32_t op, int32_t n_layers, int32_t n_q_heads, int32_t kv_heads, int32_t d,
                              int32_t cap) {
    if (n_layers < 1 || kv_heads < 1 || d < 1 || cap < 1) return 0;
    if (op == VZ_OP_DECODE) {
        if (n_q_heads < 1) return 0;
        return vz_decode_ws_bytes(n_layers, n_q_heads, kv_heads, d, cap, 0);
    }
    if (op == VZ_OP_EVICT) return vz_evict_ws_bytes(n_layers, cap, 0);
    if (op == VZ_OP_DECODE_EVICT) {
        if (n_q_heads < 1) return 0;
        return decode_evict_split(n_layers, n_q_heads, kv_heads, d, cap) + vz_evict_ws_bytes(n_layers, cap, 0);
    }
    return 0;
}

size_t voxzip_workspace_bytes_ragged(int32_t op, int32_t n_layers, int32_t n_q_heads, int32_t kv_heads, int32_t d,
                                     int64_t total, int32_t n_seqs) {
    if (n_layers < 1 || kv_heads < 1 || d < 1 || total < 1 || total > kRaggedMaxTotal) return 0;
    if (n_seqs < 1 || n_seqs > kRaggedMaxSeqs) return 0;
    if (op == VZ_OP_DECODE) {
        if (n_q_heads < 1) return 0;
        return vz_decode_ws_bytes(n_layers, n_q_heads, kv_heads, d, total, n_seqs);
    }
    if (op == VZ_OP_EVICT) return vz_evict_ws_bytes(n_layers, total, n_seqs);
    return 0;
}

int voxzip_build_span_offsets(const int64_t* t_start_ms, const int64_t* t_end_ms, const float* conf,
                              const int32_t* text_len, int32_t n_seg, int64_t t_total_ms, int32_t L_a,
                              float conf_threshold, int32_t* off_out, int32_t* n_spans_out) {
    static const char* fn = "voxzip_build_span_offsets";
    if (!off_out || !n_spans_out) return fail(VZ_ERR_INVALID, fn, "null output pointer");
    if (n_seg < 0 || t_total_ms <= 0 || L_a < 0)
        return fail(VZ_ERR_INVALID, fn, "n_seg and L_a must be >= 0 and t_total_ms > 0");
    if (n_seg > 0 && (!t_start_ms || !t_end_ms || !conf || !text_len))
        return fail(VZ_ERR_INVALID, fn, "null segment array");
    if (L_a > 0 && t_total_ms > INT64_MAX / L_a) return fail(VZ_ERR_INVALID, fn, "L_a * t_total_ms overflows");
    *n_spans_out = vz_build_span_offsets(t_start_ms, t_end_ms, conf, text_len, n_seg, t_total_ms, L_a,
                                         conf_threshold, off_out);
    return VZ_OK;
}

int voxzip_fuse_spans(const void* k_in, const void* v_in, int32_t T_in, const int32_t* span_off, int32_t n_spans,
                      const void* anchor_k, const void* anchor_v, void* k_out, void* v_out, float* score_out,
                      int32_t* pos_out, int32_t n_layers, int32_t kv_heads, int32_t d, int32_t cap_out,
                      int32_t dtype, void* stream) {
    static const char* fn = "voxzip_fuse_spans";
    if (!k_in || !span_off || !k_out || !score_out || !pos_out) return fail(VZ_ERR_INVALID, fn, "null pointer");
    int rc = check_fuse_pointers(fn, v_in, v_out, anchor_k, anchor_v);
    if (rc) return rc;
    rc = check_common(fn, n_layers, kv_heads, d, dtype, true);
    if (rc) return rc;
    if (2 * static_cast<int64_t>(kv_heads) > 65535) return fail(VZ_ERR_UNSUPPORTED, fn, "too many KV heads");
    if (T_in < 0 || n_spans < 0 || cap_out < 1) return fail(VZ_ERR_SHAPE, fn, "negative size");
    if (n_spans > T_in) return fail(VZ_ERR_SHAPE, fn, "more spans than input tokens");
    if (n_spans > cap_out) return fail(VZ_ERR_CAPACITY, fn, "n_spans exceeds cap_out");
    const size_t es = elem_size(dtype);
    const size_t in_bytes = static_cast<size_t>(n_layers) * kv_heads * T_in * d * es;
    const size_t out_bytes = static_cast<size_t>(n_layers) * kv_heads * cap_out * d * es;
    const void* ins[2] = {k_in, v_in};
    void* outs[2] = {k_out, v_out};
    for (const void* i : ins)
        for (void* o : outs)
            if (i && o && in_bytes && overlaps(i, in_bytes, o, out_bytes))
                return fail(VZ_ERR_INVALID, fn, "an input aliases an output");
    if (v_out && overlaps(k_out, out_bytes, v_out, out_bytes))
        return fail(VZ_ERR_INVALID, fn, "k_out and v_out overlap");
    hipError_t e = vz_launch_fuse(k_in, v_in, T_in, span_off, n_spans, anchor_k, anchor_v, k_out, v_out, score_out,
                                  pos_out, n_layers, kv_heads, d, cap_out, dtype, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? VZ_OK : hip_fail(fn, e);
}

int voxzip_decode_attend_score(const void* q, const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                               float* score, int32_t* pos, void* out, int32_t len, int32_t next_pos, float gamma,
                               float sm_scale, int32_t n_layers, int32_t n_q_heads, int32_t kv_heads, int32_t d,
                               int32_t cap, int32_t dtype, void* workspace, size_t ws_bytes, void* stream) {
    static const char* fn = "voxzip_decode_attend_score";
    int rc = check_decode(fn, q, k_new, v_new, k_cache, v_cache, score, pos, out, len, next_pos, gamma, sm_scale,
                          n_layers, n_q_heads, kv_heads, d, cap, dtype);
    if (rc) return rc;
    const size_t need = vz_decode_ws_bytes(n_layers, n_q_heads, kv_heads, d, cap, 0);
    if (!ws_ok(workspace, ws_bytes, need)) return fail(VZ_ERR_WORKSPACE, fn, "workspace missing, misaligned or too small");
    VzDecodeArgs a{q, k_new, v_new, k_cache, v_cache, score, pos, out, len, next_pos, gamma, sm_scale,
                   n_layers, n_q_heads, kv_heads, d, cap, dtype, workspace, ws_bytes, VzRagged{},
                   0, 0, 0, 0, nullptr, nullptr};
    hipError_t e = vz_launch_decode(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? VZ_OK : hip_fail(fn, e);
}

int voxzip_evict_compact(void* k_cache, void* v_cache, float* score, int32_t* pos, int32_t len, int32_t budget,
                         int32_t n_sink, int32_t n_recent, int32_t next_pos, int32_t* kept_pos_out,
                         int32_t* new_len_out, int32_t n_layers, int32_t kv_heads, int32_t d, int32_t cap,
                         int32_t dtype, void* workspace, size_t ws_bytes, void* stream) {
    static const char* fn = "voxzip_evict_compact";
    if (!k_cache || !v_cache || !score || !pos || !new_len_out) return fail(VZ_ERR_INVALID, fn, "null pointer");
    int rc = check_common(fn, n_layers, kv_heads, d, dtype);
    if (rc) return rc;
    int32_t M = 0;
    rc = check_evict(fn, len, budget, n_sink, n_recent, next_pos, kept_pos_out, cap, M);
    if (rc) return rc;
    const bool work = len > budget || kept_pos_out != nullptr;
    if (work) {
        const size_t need = vz_evict_ws_bytes(n_layers, cap, 0);
        if (!ws_ok(workspace, ws_bytes, need)) return fail(VZ_ERR_WORKSPACE, fn, "workspace missing, misaligned or too small");
    }
    *new_len_out = len < budget ? len : budget;
    if (!work) return VZ_OK;
    VzEvictArgs a{k_cache, v_cache, score, pos, len, budget, n_sink, M, next_pos, kept_pos_out,
                  n_layers, kv_heads, d, cap, dtype, workspace, ws_bytes, VzRagged{}, nullptr};
    hipError_t e = vz_launch_evict(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? VZ_OK : hip_fail(fn, e);
}

}  // extern "C"

namespace {

// Host checks of a generation step (both entry points); M receives the recent
// window and need the workspace bytes.
int check_step(const char* fn, const void* q, const void* k_new, const void* v_new, const void* k_cache,
               const void* v_cache, const float* score, const int32_t* pos, const void* out, int32_t len,
               int32_t next_pos, float gamma, float sm_scale, int32_t budget, int32_t n_sink, int32_t n_recent,
               const int32_t* kept_pos_out, const int32_t* new_len_out, int32_t n_layers, int32_t n_q_heads,
               int32_t kv_heads, int32_t d, int32_t cap, int32_t dtype, int32_t& M, size_t& need) {
    int rc = check_decode(fn, q, k_new, v_new, k_cache, v_cache, score, pos, out, len, next_pos, gamma, sm_scale,
                          n_layers, n_q_heads, kv_heads, d, cap, dtype);
    if (rc) return rc;
    if (!new_len_out) return fail(VZ_ERR_INVALID, fn, "null pointer");
    // the eviction sees the cache after the append
    if (next_pos == INT32_MAX) return fail(VZ_ERR_INVALID, fn, "next_pos + 1 overflows");
    rc = check_evict(fn, len + 1, budget, n_sink, n_recent, next_pos + 1, kept_pos_out, cap, M);
    if (rc) return rc;
    need = decode_evict_split(n_layers, n_q_heads, kv_heads, d, cap) + vz_evict_ws_bytes(n_layers, cap, 0);
    return VZ_OK;
}

// The generation step's launches, arguments checked (workspace of ws_bytes >= need).
int launch_step(const char* fn, const void* q, const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                float* score, int32_t* pos, void* out, int32_t len, int32_t next_pos, float gamma, float sm_scale,
                int32_t budget, int32_t n_sink, int32_t M, int32_t* kept_pos_out, int32_t* new_len_out,
                int32_t n_layers, int32_t n_q_heads, int32_t kv_heads, int32_t d, int32_t cap, int32_t dtype,
                void* workspace, size_t ws_bytes, void* stream) {
    const int32_t T = len + 1;
    const size_t split = decode_evict_split(n_layers, n_q_heads, kv_heads, d, cap);
    hipStream_t st = static_cast<hipStream_t>(stream);
    VzDecodeArgs da{q, k_new, v_new, k_cache, v_cache, score, pos, out, len, next_pos, gamma, sm_scale,
                    n_layers, n_q_heads, kv_heads, d, cap, dtype, workspace, split, VzRagged{},
                    0, 0, 0, 0, nullptr, nullptr};
    void* ews = static_cast<uint8_t*>(workspace) + split;
    VzEvictArgs ea{k_cache, v_cache, score, pos, T, budget, n_sink, M, next_pos + 1, kept_pos_out,
                   n_layers, kv_heads, d, cap, dtype, ews, ws_bytes - split, VzRagged{}, nullptr};
    const bool evict = T > budget || kept_pos_out != nullptr;
    hipError_t e;
    if (evict && vz_decode_evicts(da, budget)) {
        // one launch: the decode kernel's last workgroup per layer folds and evicts
        da.ev = 1;
        da.ev_budget = budget;
        da.ev_sink = n_sink;
        da.ev_M = M;
        da.ev_kept = kept_pos_out;
        da.ev_n = static_cast<int32_t*>(ews);  // the eviction workspace's move counts
        e = vz_launch_decode(da, st);
    } else {
        e = vz_launch_decode(da, st);
        if (e == hipSuccess && evict) e = vz_launch_evict(ea, st);
    }
    if (e != hipSuccess) return hip_fail(fn, e);
    *new_len_out = T < budget ? T : budget;
    return VZ_OK;
}

// Device address of `scratch` on the current device, looked up once per
// device (each GPU holds its own copy of the array).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices];

int scratch_address(const char* fn, void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(fn, e);
    if (dev < 0 || dev >= kMaxDevices) return fail(VZ_ERR_UNSUPPORTED, fn, "device index beyond 63");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_dev[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(fn, e);
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return VZ_OK;
}

}  // namespace

extern "C" {

int voxzip_decode_evict(const void* q, const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                        float* score, int32_t* pos, void* out, int32_t len, int32_t next_pos, float gamma,
                        float sm_scale, int32_t budget, int32_t n_sink, int32_t n_recent, int32_t* kept_pos_out,
                        int32_t* new_len_out, int32_t n_layers, int32_t n_q_heads, int32_t kv_heads, int32_t d,
                        int32_t cap, int32_t dtype, void* workspace, size_t ws_bytes, void* stream) {
    static const char* fn = "voxzip_decode_evict";
    int32_t M = 0;
    size_t need = 0;
    int rc = check_step(fn, q, k_new, v_new, k_cache, v_cache, score, pos, out, len, next_pos, gamma, sm_scale, budget,
                        n_sink, n_recent, kept_pos_out, new_len_out, n_layers, n_q_heads, kv_heads, d, cap, dtype, M,
                        need);
    if (rc) return rc;
    if (!ws_ok(workspace, ws_bytes, need)) return fail(VZ_ERR_WORKSPACE, fn, "workspace missing, misaligned or too small");
    return launch_step(fn, q, k_new, v_new, k_cache, v_cache, score, pos, out, len, next_pos, gamma, sm_scale, budget,
                       n_sink, M, kept_pos_out, new_len_out, n_layers, n_q_heads, kv_heads, d, cap, dtype, workspace,
                       ws_bytes, stream);
}

int voxzip_decode_evict_noalloc(const void* q, const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                                float* score, int32_t* pos, void* out, int32_t len, int32_t next_pos, float gamma,
                                float sm_scale, int32_t budget, int32_t n_sink, int32_t n_recent,
                                int32_t* kept_pos_out, int32_t* new_len_out, int32_t n_layers, int32_t n_q_heads,
                                int32_t kv_heads, int32_t d, int32_t cap, int32_t dtype, void* stream) {
    static const char* fn = "voxzip_decode_evict_noalloc";
    int32_t M = 0;
    size_t need = 0;
    int rc = check_step(fn, q, k_new, v_new, k_cache, v_cache, score, pos, out, len, next_pos, gamma, sm_scale, budget,
                        n_sink, n_recent, kept_pos_out, new_len_out, n_layers, n_q_heads, kv_heads, d, cap, dtype, M,
                        need);
    if (rc) return rc;
    if (need > VZ_NOALLOC_SCRATCH_BYTES) {
        g_last_error = std::string(fn) + ": the call needs " + std::to_string(need) +
                       " bytes of scratch memory (voxzip_workspace_bytes(VZ_OP_DECODE_EVICT, ...)); this entry point "
                       "holds " + std::to_string(static_cast<size_t>(VZ_NOALLOC_SCRATCH_BYTES)) +
                       ": use voxzip_decode_evict with a workspace";
        return VZ_ERR_WORKSPACE;
    }
    void* ws = nullptr;
    rc = scratch_address(fn, &ws);
    if (rc) return rc;
    return launch_step(fn, q, k_new, v_new, k_cache, v_cache, score, pos, out, len, next_pos, gamma, sm_scale, budget,
                       n_sink, M, kept_pos_out, new_len_out, n_layers, n_q_heads, kv_heads, d, cap, dtype, ws,
                       VZ_NOALLOC_SCRATCH_BYTES, stream);
}

int voxzip_fuse_spans_ragged(const void* k_in, const void* v_in, const int64_t* in_base, const int32_t* T_in,
                             int64_t total_in, const int32_t* span_off, const int64_t* off_base,
                             const int32_t* n_spans, int64_t total_off, int32_t max_spans, const void* anchor_k,
                             const void* anchor_v, void* k_out, void* v_out, float* score_out, int32_t* pos_out,
                             const int64_t* seq_base, const int32_t* cap, int64_t total, int32_t n_seqs,
                             int32_t* status, int32_t n_layers, int32_t kv_heads, int32_t d, int32_t dtype,
                             void* stream) {
    static const char* fn = "voxzip_fuse_spans_ragged";
    if (!k_in || !in_base || !T_in || !span_off || !off_base || !n_spans || !k_out || !score_out || !pos_out ||
        !seq_base || !cap)
        return fail(VZ_ERR_INVALID, fn, "null pointer");
    int rc = check_fuse_pointers(fn, v_in, v_out, anchor_k, anchor_v);
    if (rc) return rc;
    rc = check_ragged(fn, n_layers, kv_heads, d, dtype, total, n_seqs, true);
    if (rc) return rc;
    if (total_in < 0 || total_off < 1 || max_spans < 0) return fail(VZ_ERR_SHAPE, fn, "negative size");
    if (total_in > kRaggedMaxTotal || max_spans > total) return fail(VZ_ERR_SHAPE, fn, "size out of range");
    if (2 * static_cast<int64_t>(kv_heads) > 65535) return fail(VZ_ERR_UNSUPPORTED, fn, "too many KV heads");
    if (static_cast<int64_t>(max_spans > 0 ? max_spans : 1) * n_seqs >= (int64_t(1) << 31))
        return fail(VZ_ERR_UNSUPPORTED, fn, "max_spans x n_seqs too large");
    const size_t es = elem_size(dtype);
    const size_t in_bytes = static_cast<size_t>(n_layers) * kv_heads * total_in * d * es;
    const size_t out_bytes = static_cast<size_t>(n_layers) * kv_heads * total * d * es;
    const void* ins[2] = {k_in, v_in};
    void* outs[2] = {k_out, v_out};
    for (const void* i : ins)
        for (void* o : outs)
            if (i && o && in_bytes && overlaps(i, in_bytes, o, out_bytes))
                return fail(VZ_ERR_INVALID, fn, "an input aliases an output");
    if (v_out && overlaps(k_out, out_bytes, v_out, out_bytes))
        return fail(VZ_ERR_INVALID, fn, "k_out and v_out overlap");
    VzFuseRaggedArgs a{k_in,     v_in,     in_base,  T_in,     span_off, off_base,  n_spans,  anchor_k,
                       anchor_v, k_out,    v_out,    score_out, pos_out, seq_base,  cap,      status,
                       n_seqs,   total_in, total_off, total,   max_spans, n_layers, kv_heads, d,
                       dtype};
    hipError_t e = vz_launch_fuse_ragged(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? VZ_OK : hip_fail(fn, e);
}

int voxzip_decode_attend_score_ragged(const void* q, const void* k_new, const void* v_new, void* k_cache,
                                      void* v_cache, float* score, int32_t* pos, void* out, const int64_t* seq_base,
                                      const int32_t* cap, const int32_t* len, const int32_t* next_pos, int64_t total,
                                      int32_t n_seqs, float gamma, float sm_scale, int32_t n_layers,
                                      int32_t n_q_heads, int32_t kv_heads, int32_t d, int32_t dtype,
                                      int32_t* status, void* workspace, size_t ws_bytes, void* stream) {
    static const char* fn = "voxzip_decode_attend_score_ragged";
    if (!q || !k_new || !v_new || !k_cache || !v_cache || !score || !pos || !out || !seq_base || !cap || !len ||
        !next_pos)
        return fail(VZ_ERR_INVALID, fn, "null pointer");
    int rc = check_ragged(fn, n_layers, kv_heads, d, dtype, total, n_seqs);
    if (rc) return rc;
    if (n_q_heads < 1 || n_q_heads % kv_heads != 0)
        return fail(VZ_ERR_SHAPE, fn, "n_q_heads must be a positive multiple of kv_heads");
    if (n_q_heads / kv_heads > 16) return fail(VZ_ERR_UNSUPPORTED, fn, "more than 16 query heads per KV head");
    if (n_q_heads > 256) return fail(VZ_ERR_UNSUPPORTED, fn, "more than 256 query heads");
    if (!(gamma >= 0.f && gamma <= 1.f)) return fail(VZ_ERR_INVALID, fn, "gamma must be in [0, 1]");
    if (!isfinite(sm_scale)) return fail(VZ_ERR_INVALID, fn, "sm_scale must be finite");
    const size_t need = vz_decode_ws_bytes(n_layers, n_q_heads, kv_heads, d, total, n_seqs);
    if (!ws_ok(workspace, ws_bytes, need)) return fail(VZ_ERR_WORKSPACE, fn, "workspace missing, misaligned or too small");
    VzRagged rg{seq_base, cap, len, next_pos, nullptr, status, n_seqs, total};
    VzDecodeArgs a{q,  k_new, v_new, k_cache, v_cache, score, pos,   out,       0,        0,  gamma, sm_scale,
                   n_layers, n_q_heads, kv_heads, d, 0, dtype, workspace, ws_bytes, rg,
                   0, 0, 0, 0, nullptr, nullptr};
    hipError_t e = vz_launch_decode(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? VZ_OK : hip_fail(fn, e);
}

int voxzip_evict_compact_ragged(void* k_cache, void* v_cache, float* score, int32_t* pos, const int64_t* seq_base,
                                const int32_t* cap, const int32_t* len, const int32_t* budget,
                                const int32_t* next_pos, int64_t total, int32_t n_seqs, int32_t n_sink,
                                int32_t n_recent, int32_t* kept_pos_out, int32_t* new_len_out, int32_t* status,
                                int32_t n_layers, int32_t kv_heads, int32_t d, int32_t dtype, void* workspace,
                                size_t ws_bytes, void* stream) {
    static const char* fn = "voxzip_evict_compact_ragged";
    if (!k_cache || !v_cache || !score || !pos || !seq_base || !cap || !len || !budget || !next_pos)
        return fail(VZ_ERR_INVALID, fn, "null pointer");
    int rc = check_ragged(fn, n_layers, kv_heads, d, dtype, total, n_seqs);
    if (rc) return rc;
    if (n_sink < 0) return fail(VZ_ERR_INVALID, fn, "n_sink must be >= 0");
    if (new_len_out && overlaps(new_len_out, 4 * static_cast<size_t>(n_seqs), len, 4 * static_cast<size_t>(n_seqs)))
        return fail(VZ_ERR_INVALID, fn, "new_len_out must not overlap len");
    const size_t need = vz_evict_ws_bytes(n_layers, total, n_seqs);
    if (!ws_ok(workspace, ws_bytes, need)) return fail(VZ_ERR_WORKSPACE, fn, "workspace missing, misaligned or too small");
    VzRagged rg{seq_base, cap, len, next_pos, budget, status, n_seqs, total};
    VzEvictArgs a{k_cache, v_cache, score, pos, 0, 0, n_sink, n_recent, 0, kept_pos_out,
                  n_layers, kv_heads, d, 0, dtype, workspace, ws_bytes, rg, new_len_out};
    hipError_t e = vz_launch_evict(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? VZ_OK : hip_fail(fn, e);
}

}  // extern "C"

size_t vz_decode_ws_bytes(int32_t L, int32_t Hq, int32_t Hkv, int32_t d, int64_t plane, int32_t n_seqs) {
    (void)d;
    const size_t gen = vz_decode_generic_ws_bytes(L, Hq, plane, n_seqs);
    const size_t fused = vz_decode_fused_ws_bytes(L, Hq, plane, n_seqs);
    const size_t range = Hkv > 0 && Hq % Hkv == 0 ? vz_decode_range_ws_bytes(L, Hq, Hkv, plane, n_seqs) : 0;
    return std::max(std::max(gen, fused), range);
}

hipError_t vz_launch_decode(const VzDecodeArgs& a, hipStream_t stream) {
    const int64_t plane = a.rag.n > 0 ? a.rag.total : a.cap;
    if (vz_decode_fused_ok(a.dtype, a.d, a.Hq, a.Hkv, a.L, plane, a.rag.n)) return vz_launch_decode_fused(a, stream);
    if (!vz_decode_generic_ok(plane, a.rag.n)) return hipErrorInvalidValue;
    return vz_launch_decode_generic(a, stream);
}
