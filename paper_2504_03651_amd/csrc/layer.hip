// layer.hip -- one decoder layer around the mixed iteration (include/echo_layer.h):
// element-wise kernels for gfx950 (RMSNorm, RoPE + split, SiLU * up, fp32 ->
// bf16) and the hipBLASLt GEMMs, then echo_kv_append / echo_attn_mixed.
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>
#include <tuple>

#include "echo_layer.h"
#include "status.hpp"

namespace {

using echo::fail;

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest even (NaN stays a quiet NaN)
__device__ __forceinline__ uint16_t f2bf(float x) {
    const uint32_t u = __float_as_uint(x);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// One workgroup per token row: y = x / sqrt(mean(x^2) + eps) * w, fp32 math.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const uint16_t *x, const uint16_t *w,
                                                      uint16_t *y, int H, float eps) {
    const int64_t row = blockIdx.x;
    const uint16_t *xr = x + row * H;
    uint16_t *yr = y + row * H;
    float ss = 0.f;
    for (int c = threadIdx.x * 8; c < H; c += 256 * 8) {
        const u32x4 v = *(const u32x4 *)(xr + c);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = bf2f((uint16_t)(v[e] & 0xFFFF)), b = bf2f((uint16_t)(v[e] >> 16));
            ss += a * a + b * b;
        }
    }
    __shared__ float part[4];
    for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float tot = part[0] + part[1] + part[2] + part[3];
    const float inv = 1.f / sqrtf(tot / (float)H + eps);
    for (int c = threadIdx.x * 8; c < H; c += 256 * 8) {
        const u32x4 v = *(const u32x4 *)(xr + c);
        const u32x4 g = *(const u32x4 *)(w + c);
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = bf2f((uint16_t)(v[e] & 0xFFFF)) * inv * bf2f((uint16_t)(g[e] & 0xFFFF));
            const float b = bf2f((uint16_t)(v[e] >> 16)) * inv * bf2f((uint16_t)(g[e] >> 16));
            o[e] = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
        }
        *(u32x4 *)(yr + c) = o;
    }
}

// One workgroup per token: its position from the batch (binary search over
// q_start), the rotation angles of its D/2 frequency pairs in fp64 (shared by
// all heads through LDS), then q and k heads rotated and v copied out of qkv.
__global__ __launch_bounds__(256) void rope_split_kernel(
    const uint16_t *qkv, const int32_t *q_start, const int32_t *seq_lens, int B, int Hq, int Hkv,
    int D, double log2_theta, uint16_t *q, uint16_t *k, uint16_t *v) {
    const int t = blockIdx.x;
    int lo = 0, hi = B;   // row r with q_start[r] <= t < q_start[r + 1]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (q_start[mid] <= t) lo = mid;
        else hi = mid;
    }
    const int r = lo;
    const int pos = seq_lens[r] - (q_start[r + 1] - q_start[r]) + (t - q_start[r]);
    __shared__ float cs[2][128];   // cos, sin of the D/2 <= 128 pairs
    const int half = D / 2;
    for (int i = threadIdx.x; i < half; i += 256) {
        const double ang = (double)pos * exp2(-(double)(2 * i) / (double)D * log2_theta);
        double sn, cn;
        sincos(ang, &sn, &cn);
        cs[0][i] = (float)cn;
        cs[1][i] = (float)sn;
    }
    __syncthreads();
    const int W = (Hq + 2 * Hkv) * D;
    const uint16_t *src = qkv + (int64_t)t * W;
    const int npairs = (Hq + Hkv) * half;
    for (int e = threadIdx.x; e < npairs; e += 256) {
        const int h = e / half, i = e - h * half;
        const float x1 = bf2f(src[h * D + i]), x2 = bf2f(src[h * D + i + half]);
        const float c = cs[0][i], s = cs[1][i];
        const uint16_t o1 = f2bf(x1 * c - x2 * s), o2 = f2bf(x2 * c + x1 * s);
        uint16_t *dst = h < Hq ? q + ((int64_t)t * Hq + h) * D : k + ((int64_t)t * Hkv + (h - Hq)) * D;
        dst[i] = o1;
        dst[i + half] = o2;
    }
    for (int e = threadIdx.x; e < Hkv * D; e += 256) v[(int64_t)t * Hkv * D + e] = src[(Hq + Hkv) * D + e];
}

__global__ __launch_bounds__(256) void f32_to_bf16_kernel(const float *x, uint16_t *y, int64_t n4) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n4) return;
    const float4 a = ((const float4 *)x)[i];
    uint2 o;
    o.x = (uint32_t)f2bf(a.x) | ((uint32_t)f2bf(a.y) << 16);
    o.y = (uint32_t)f2bf(a.z) | ((uint32_t)f2bf(a.w) << 16);
    ((uint2 *)y)[i] = o;
}

// act[t][j] = SiLU(gate) * up with gate = gu[t][j], up = gu[t][I + j], fp32 math
__global__ __launch_bounds__(256) void silu_mul_kernel(const uint16_t *gu, uint16_t *act, int I,
                                                       int64_t n8) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n8) return;
    const int64_t e = i * 8, t = e / I, j = e - t * I;
    const u32x4 g = *(const u32x4 *)(gu + t * 2 * I + j);
    const u32x4 u = *(const u32x4 *)(gu + t * 2 * I + I + j);
    u32x4 o;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const float g0 = bf2f((uint16_t)(g[c] & 0xFFFF)), g1 = bf2f((uint16_t)(g[c] >> 16));
        const float u0 = bf2f((uint16_t)(u[c] & 0xFFFF)), u1 = bf2f((uint16_t)(u[c] >> 16));
        const float a0 = g0 / (1.f + expf(-g0)) * u0, a1 = g1 / (1.f + expf(-g1)) * u1;
        o[c] = (uint32_t)f2bf(a0) | ((uint32_t)f2bf(a1) << 16);
    }
    *(u32x4 *)(act + e) = o;
}

// ------------------------------------------------------------------ hipBLASLt

// Y [T][N] (+ R [T][N]) = X [T][K] W[N][K]^T, row-major bf16, fp32 accumulate:
// column-major D (N x T) = op(A) B with A = W seen as K x N (transposed),
// B = X seen as K x T.
struct GemmPlan {
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
    hipblasLtMatmulAlgo_t algo{};
    size_t ws = 0;
};

struct Blas {
    hipblasLtHandle_t h = nullptr;
    std::map<std::tuple<int64_t, int64_t, int64_t, bool>, GemmPlan> plans;
};

constexpr size_t kBlasWs = 32u << 20;

int blas_fail(hipblasStatus_t s, const char *what) {
    return fail(ECHO_E_HIP, "%s: hipBLASLt status %d", what, (int)s);
}

int get_blas(Blas **out) {
    thread_local std::map<int, Blas> per_dev;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(ECHO_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    Blas &b = per_dev[dev];
    if (!b.h) {
        hipblasStatus_t s = hipblasLtCreate(&b.h);
        if (s != HIPBLAS_STATUS_SUCCESS) {
            b.h = nullptr;
            return blas_fail(s, "hipblasLtCreate");
        }
    }
    *out = &b;
    return ECHO_OK;
}

int gemm(Blas *bl, int64_t N, int64_t T, int64_t K, const void *W, const void *X,
         const void *R, void *Y, void *ws, hipStream_t st) {
    const bool acc = R != nullptr;
    auto key = std::make_tuple(N, T, K, acc);
    auto it = bl->plans.find(key);
    hipblasStatus_t s;
    if (it == bl->plans.end() && bl->plans.size() >= 256) {   // token counts vary per call
        for (auto &kv : bl->plans) {
            hipblasLtMatrixLayoutDestroy(kv.second.a);
            hipblasLtMatrixLayoutDestroy(kv.second.b);
            hipblasLtMatrixLayoutDestroy(kv.second.c);
            hipblasLtMatmulDescDestroy(kv.second.desc);
        }
        bl->plans.clear();
    }
    if (it == bl->plans.end()) {
        GemmPlan p;
        if ((s = hipblasLtMatmulDescCreate(&p.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F)) !=
            HIPBLAS_STATUS_SUCCESS)
            return blas_fail(s, "hipblasLtMatmulDescCreate");
        const int32_t opT = HIPBLAS_OP_T, opN = HIPBLAS_OP_N;
        hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opT, sizeof opT);
        hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opN, sizeof opN);
        if ((s = hipblasLtMatrixLayoutCreate(&p.a, HIP_R_16BF, K, N, K)) != HIPBLAS_STATUS_SUCCESS ||
            (s = hipblasLtMatrixLayoutCreate(&p.b, HIP_R_16BF, K, T, K)) != HIPBLAS_STATUS_SUCCESS ||
            (s = hipblasLtMatrixLayoutCreate(&p.c, HIP_R_16BF, N, T, N)) != HIPBLAS_STATUS_SUCCESS)
            return blas_fail(s, "hipblasLtMatrixLayoutCreate");
        hipblasLtMatmulPreference_t pref;
        if ((s = hipblasLtMatmulPreferenceCreate(&pref)) != HIPBLAS_STATUS_SUCCESS)
            return blas_fail(s, "hipblasLtMatmulPreferenceCreate");
        const uint64_t max_ws = kBlasWs;
        hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES,
                                              &max_ws, sizeof max_ws);
        hipblasLtMatmulHeuristicResult_t res{};
        int n = 0;
        s = hipblasLtMatmulAlgoGetHeuristic(bl->h, p.desc, p.a, p.b, p.c, p.c, pref, 1, &res, &n);
        hipblasLtMatmulPreferenceDestroy(pref);
        if (s != HIPBLAS_STATUS_SUCCESS || n < 1)
            return fail(ECHO_E_HIP, "no hipBLASLt algorithm for %lld x %lld x %lld", (long long)N,
                        (long long)T, (long long)K);
        p.algo = res.algo;
        p.ws = res.workspaceSize;
        it = bl->plans.emplace(key, p).first;
    }
    const GemmPlan &p = it->second;
    const float alpha = 1.f, beta = acc ? 1.f : 0.f;
    s = hipblasLtMatmul(bl->h, p.desc, &alpha, W, p.a, X, p.b, &beta, acc ? R : Y, p.c, Y, p.c,
                        &p.algo, ws, std::min(p.ws, kBlasWs), st);
    if (s != HIPBLAS_STATUS_SUCCESS) return blas_fail(s, "hipblasLtMatmul");
    return ECHO_OK;
}

// ------------------------------------------------------------------ layout

struct Ws {
    size_t y, qkv, q, kn, vn, attn, attn_ws, attn16, h, gu, act, blas, total;
};

size_t up256(size_t x) { return (x + 255) / 256 * 256; }

int plan_ws(const echo_layer_t *L, const echo_kv_pool_t *pool, const echo_batch_t *b, Ws *w) {
    if (!L || !pool || !b) return fail(ECHO_E_INVALID, "layer, pool or batch is NULL");
    if (L->hidden <= 0 || L->hidden % 8 || L->intermediate <= 0 || L->intermediate % 8 ||
        L->num_q_heads <= 0 || L->num_kv_heads <= 0 || L->num_q_heads % L->num_kv_heads)
        return fail(ECHO_E_INVALID, "layer shape (H %d, I %d, Hq %d, Hkv %d)", L->hidden,
                    L->intermediate, L->num_q_heads, L->num_kv_heads);
    if (L->head_dim != pool->head_dim || L->num_kv_heads != pool->num_kv_heads)
        return fail(ECHO_E_INVALID, "layer heads (%d x %d) differ from the pool's (%d x %d)",
                    L->num_kv_heads, L->head_dim, pool->num_kv_heads, pool->head_dim);
    if (L->head_dim > 256 || L->head_dim % 2)
        return fail(ECHO_E_UNSUPPORTED, "head_dim %d", L->head_dim);
    if (!L->attn_norm || !L->w_qkv || !L->w_o || !L->mlp_norm || !L->w_gate_up || !L->w_down)
        return fail(ECHO_E_INVALID, "a layer weight is NULL");
    int rc = echo_validate(pool, b, 1);
    if (rc) return rc;
    const int64_t T = b->num_tokens, H = L->hidden, I = L->intermediate;
    const int64_t qd = (int64_t)L->num_q_heads * L->head_dim;
    const int64_t kd = (int64_t)L->num_kv_heads * L->head_dim;
    const size_t attn_ws = echo_attn_workspace_bytes(pool, b, L->num_q_heads);
    if (attn_ws == 0 && b->num_rows > 0) return ECHO_E_INVALID;   // detail already set
    size_t o = 0;
    auto take = [&](size_t n) { const size_t at = o; o += up256(n); return at; };
    w->y = take(T * H * 2);
    w->qkv = take(T * (qd + 2 * kd) * 2);
    w->q = take(T * qd * 2);
    w->kn = take(T * kd * 2);
    w->vn = take(T * kd * 2);
    w->attn = take(T * qd * 4);
    w->attn_ws = take(std::max<size_t>(attn_ws, 256));
    w->attn16 = take(T * qd * 2);
    w->h = take(T * H * 2);
    w->gu = take(T * 2 * I * 2);
    w->act = take(T * I * 2);
    w->blas = take(kBlasWs);
    w->total = o;
    return ECHO_OK;
}

struct LayerProfile {
    int device = -1;
    hipEvent_t ev[12] = {};
    bool valid = false;
};
thread_local LayerProfile g_lprof;

}  // namespace

extern "C" {

size_t echo_layer_workspace_bytes(const echo_layer_t *layer, const echo_kv_pool_t *pool,
                                  const echo_batch_t *batch) {
    echo::clear_error();
    Ws w;
    if (plan_ws(layer, pool, batch, &w)) return 0;
    return w.total;
}

int echo_layer_forward(const echo_layer_t *L, const echo_kv_pool_t *pool,
                       const echo_batch_t *batch, void *hidden, void *workspace,
                       size_t workspace_bytes, void *host_workspace,
                       size_t host_workspace_bytes, void *stream) {
    echo::clear_error();
    Ws w;
    int rc = plan_ws(L, pool, batch, &w);
    if (rc) return rc;
    if (batch->num_rows == 0) return ECHO_OK;
    if (!hidden) return fail(ECHO_E_INVALID, "hidden is NULL");
    if (!workspace || workspace_bytes < w.total || ((uintptr_t)workspace & 255u))
        return fail(ECHO_E_WORKSPACE, "workspace of %zu bytes (need %zu, 256-byte aligned)",
                    workspace_bytes, w.total);
    Blas *bl = nullptr;
    if ((rc = get_blas(&bl))) return rc;
    hipStream_t st = (hipStream_t)stream;
    uint8_t *base = (uint8_t *)workspace;
    uint16_t *y = (uint16_t *)(base + w.y), *qkv = (uint16_t *)(base + w.qkv);
    uint16_t *q = (uint16_t *)(base + w.q), *kn = (uint16_t *)(base + w.kn);
    uint16_t *vn = (uint16_t *)(base + w.vn), *a16 = (uint16_t *)(base + w.attn16);
    uint16_t *h = (uint16_t *)(base + w.h), *gu = (uint16_t *)(base + w.gu);
    uint16_t *act = (uint16_t *)(base + w.act);
    float *attn = (float *)(base + w.attn);
    void *bws = base + w.blas;
    uint16_t *x = (uint16_t *)hidden;
    const int T = batch->num_tokens, H = L->hidden, I = L->intermediate;
    const int Hq = L->num_q_heads, Hkv = L->num_kv_heads, D = L->head_dim;

    // stage events (profiling only): 0 start, then after each stage
    hipEvent_t *ev = nullptr;
    if (echo::profile_enabled()) {
        int dev = 0;
        (void)hipGetDevice(&dev);
        if (g_lprof.device != dev) {
            for (hipEvent_t &e : g_lprof.ev)
                if (e) (void)hipEventDestroy(e), e = nullptr;
            g_lprof.device = dev;
        }
        for (hipEvent_t &e : g_lprof.ev)
            if (!e && hipEventCreate(&e) != hipSuccess) return fail(ECHO_E_HIP, "hipEventCreate");
        ev = g_lprof.ev;
        g_lprof.valid = false;
    }
    auto mark = [&](int i) {
        if (ev) (void)hipEventRecord(ev[i], st);
    };
    auto check = [&](const char *what) -> int {
        hipError_t e = hipGetLastError();
        return e == hipSuccess ? ECHO_OK : fail(ECHO_E_HIP, "%s: %s", what, hipGetErrorString(e));
    };
    mark(0);
    hipLaunchKernelGGL(rmsnorm_kernel, dim3(T), dim3(256), 0, st, x, (const uint16_t *)L->attn_norm,
                       y, H, L->rms_eps);
    if ((rc = check("rmsnorm"))) return rc;
    mark(1);
    if ((rc = gemm(bl, (int64_t)(Hq + 2 * Hkv) * D, T, H, L->w_qkv, y, nullptr, qkv, bws, st))) return rc;
    mark(2);
    hipLaunchKernelGGL(rope_split_kernel, dim3(T), dim3(256), 0, st, qkv, batch->q_start,
                       batch->seq_lens, batch->num_rows, Hq, Hkv, D, std::log2((double)L->rope_theta),
                       q, kn, vn);
    if ((rc = check("rope"))) return rc;
    mark(3);
    if ((rc = echo_kv_append(pool, batch, kn, vn, stream))) return rc;
    mark(4);
    if ((rc = echo_attn_mixed(pool, batch, q, Hq, (float)(1.0 / std::sqrt((double)D)), attn,
                              base + w.attn_ws, w.attn16 - w.attn_ws, host_workspace,
                              host_workspace_bytes, stream)))
        return rc;
    mark(5);
    const int64_t n4 = (int64_t)T * Hq * D / 4;
    hipLaunchKernelGGL(f32_to_bf16_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, st,
                       attn, a16, n4);
    if ((rc = check("cast"))) return rc;
    mark(6);
    if ((rc = gemm(bl, H, T, (int64_t)Hq * D, L->w_o, a16, x, h, bws, st))) return rc;
    mark(7);
    hipLaunchKernelGGL(rmsnorm_kernel, dim3(T), dim3(256), 0, st, h, (const uint16_t *)L->mlp_norm,
                       y, H, L->rms_eps);
    if ((rc = check("rmsnorm"))) return rc;
    mark(8);
    if ((rc = gemm(bl, 2 * (int64_t)I, T, H, L->w_gate_up, y, nullptr, gu, bws, st))) return rc;
    mark(9);
    const int64_t n8 = (int64_t)T * I / 8;
    hipLaunchKernelGGL(silu_mul_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, st, gu,
                       act, I, n8);
    if ((rc = check("silu_mul"))) return rc;
    mark(10);
    if ((rc = gemm(bl, H, T, I, L->w_down, act, h, x, bws, st))) return rc;
    mark(11);
    if (ev) g_lprof.valid = true;
    return ECHO_OK;
}

int echo_layer_timing(echo_layer_timing_t *t) {
    echo::clear_error();
    if (!t) return fail(ECHO_E_INVALID, "timing is NULL");
    if (!g_lprof.valid) return fail(ECHO_E_INVALID, "no profiled echo_layer_forward on this thread");
    float ms[11];
    if (hipEventSynchronize(g_lprof.ev[11]) != hipSuccess) return fail(ECHO_E_HIP, "event");
    for (int i = 0; i < 11; ++i)
        if (hipEventElapsedTime(&ms[i], g_lprof.ev[i], g_lprof.ev[i + 1]) != hipSuccess)
            return fail(ECHO_E_HIP, "hipEventElapsedTime");
    // stages: 0 norm, 1 qkv, 2 rope, 3 append, 4 attention, 5 cast, 6 o, 7 norm,
    // 8 gate_up, 9 silu, 10 down
    t->norm_ms = ms[0] + ms[7];
    t->qkv_ms = ms[1];
    t->rope_ms = ms[2];
    t->append_ms = ms[3];
    t->attention_ms = ms[4];
    t->o_ms = ms[6];
    t->mlp_ms = ms[8] + ms[10];
    t->other_ms = ms[5] + ms[9];
    return ECHO_OK;
}

}  // extern "C"
