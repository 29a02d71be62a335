// Simple per-op kernels of the expert tick (Sec. 3.1, Eq. (1)) for any shape and for fp32 weights.
// Every value is computed in fp32 with one thread per output element; these kernels serve the fp32
// expert (whose tolerance needs fp32 arithmetic end to end) and shapes the fused bf16 path does not
// cover.  Same readings as the fused path: pre-norm RMSNorm, rotary pairs (j, j + Dh/2), scale
// 1/sqrt(Dh), SwiGLU, mean-pool head.

#include "common.h"
#include "kernels.h"

namespace fsx {

__device__ __forceinline__ float ld(const void* p, int dtype, int64_t i) {
  if (dtype == FSX_BF16) return bf16_to_f32(((const uint16_t*)p)[i]);
  if (dtype == FSX_FP8_E4M3) return e4m3_to_f32(((const uint8_t*)p)[i]);
  return ((const float*)p)[i];
}

__global__ void g_embed(const void* tokens, int dtype, TickParams tp, Dims dm, GenericWorkspace ws) {
  const int m = blockIdx.x;
  const int b = m / tp.S, t = m % tp.S;
  for (int n = threadIdx.x; n < dm.d; n += blockDim.x) ws.h[(int64_t)m * dm.d + n] = ld(tokens, dtype, (int64_t)m * dm.d + n);
  const int half = dm.Dh / 2;
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    double cs = 1.0, sn = 0.0;
    if (dm.rope_base > 0.f) {
      const double ang = (double)(tp.pos[b] + t) * pow((double)dm.rope_base, -2.0 * (double)j / (double)dm.Dh);
      cs = cos(ang);
      sn = sin(ang);
    }
    ws.rope[((int64_t)m * half + j) * 2] = (float)cs;
    ws.rope[((int64_t)m * half + j) * 2 + 1] = (float)sn;
  }
}

// x = RMSNorm(h) * g, one workgroup per row
__global__ void g_norm(const float* h, const float* g, float* x, int d, float eps) {
  __shared__ float red[16];
  const int m = blockIdx.x;
  float ss = 0.f;
  for (int n = threadIdx.x; n < d; n += blockDim.x) ss += h[(int64_t)m * d + n] * h[(int64_t)m * d + n];
  ss = block_sum(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  for (int n = threadIdx.x; n < d; n += blockDim.x) x[(int64_t)m * d + n] = h[(int64_t)m * d + n] * r * g[n];
}

// y[m][n] (+)= sum_k x[m][k] W[n][k]
__global__ void g_linear(const float* x, const void* W, int wdtype, float* y, int M, int N, int K, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * N) return;
  const int m = (int)(i / N), n = (int)(i % N);
  float acc = 0.f;
  for (int k = 0; k < K; ++k) acc += x[(int64_t)m * K + k] * ld(W, wdtype, (int64_t)n * K + k);
  y[i] = accumulate ? y[i] + acc : acc;
}

// rotate q and k in place (pairs j, j+Dh/2) and scale q by 1/sqrt(Dh)
__global__ void g_rope(float* q, float* k, const float* rope, int M, int H, int Dh) {
  const int half = Dh / 2;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * H * half) return;
  const int j = (int)(i % half);
  const int64_t mh = i / half;
  const int m = (int)(mh / H);
  const float cs = rope[((int64_t)m * half + j) * 2], sn = rope[((int64_t)m * half + j) * 2 + 1];
  const int64_t o = mh * Dh;
  const float qs = 1.0f / sqrtf((float)Dh);
  const float q1 = q[o + j], q2 = q[o + j + half], k1 = k[o + j], k2 = k[o + j + half];
  q[o + j] = (q1 * cs - q2 * sn) * qs;
  q[o + j + half] = (q2 * cs + q1 * sn) * qs;
  k[o + j] = k1 * cs - k2 * sn;
  k[o + j + half] = k2 * cs + k1 * sn;
}

// one thread per (agent, head, query token): two passes over [cache rows ; own rows]
__global__ void g_attention(CacheView cv, TickParams tp, const float* q, const float* k, const float* v, float* out,
                            int H, int Dh) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)tp.M * H) return;
  const int h = (int)(i % H);
  const int m = (int)(i / H);
  const int b = m / tp.S;
  const int A = H * Dh;
  const float* qr = q + (int64_t)m * A + (int64_t)h * Dh;
  const int L = tp.len[b];
  const int64_t hb = cache_head_base(cv, b, cv.layer, h);  // ring slot 0 of (agent, layer, head)
  float ks = 1.f, vs = 1.f;
  if (cv.dtype == FSX_FP8_E4M3) {
    ks = cv.k_scale[cache_scale_index(cv, b, cv.layer, h)];
    vs = cv.v_scale[cache_scale_index(cv, b, cv.layer, h)];
  }
  auto cache_off = [&](int r) {
    int64_t slot = tp.start[b] + r;
    if (slot >= cv.cap) slot -= cv.cap;
    return hb + slot * cv.rs;
  };
  float mx = -INFINITY;
  for (int r = 0; r < L; ++r) {
    const int64_t o = cache_off(r);
    float s = 0.f;
    for (int c = 0; c < Dh; ++c) s += qr[c] * ld(cv.k, cv.dtype, o + c);
    mx = fmaxf(mx, s * ks);
  }
  for (int r = 0; r < tp.S; ++r) {
    const float* kr = k + ((int64_t)b * tp.S + r) * A + (int64_t)h * Dh;
    float s = 0.f;
    for (int c = 0; c < Dh; ++c) s += qr[c] * kr[c];
    mx = fmaxf(mx, s);
  }
  float* o = out + (int64_t)m * A + (int64_t)h * Dh;
  for (int c = 0; c < Dh; ++c) o[c] = 0.f;
  float l = 0.f;
  for (int r = 0; r < L; ++r) {
    const int64_t off = cache_off(r);
    float s = 0.f;
    for (int c = 0; c < Dh; ++c) s += qr[c] * ld(cv.k, cv.dtype, off + c);
    const float p = expf(s * ks - mx);
    l += p;
    for (int c = 0; c < Dh; ++c) o[c] += p * vs * ld(cv.v, cv.dtype, off + c);
  }
  for (int r = 0; r < tp.S; ++r) {
    const float* kr = k + ((int64_t)b * tp.S + r) * A + (int64_t)h * Dh;
    const float* vr = v + ((int64_t)b * tp.S + r) * A + (int64_t)h * Dh;
    float s = 0.f;
    for (int c = 0; c < Dh; ++c) s += qr[c] * kr[c];
    const float p = expf(s - mx);
    l += p;
    for (int c = 0; c < Dh; ++c) o[c] += p * vr[c];
  }
  const float inv = 1.0f / l;
  for (int c = 0; c < Dh; ++c) o[c] *= inv;
}

// g = silu(g) * u
__global__ void g_swiglu(float* g, const float* u, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float x = g[i];
  g[i] = x / (1.0f + expf(-x)) * u[i];
}

__global__ void g_copy(const float* src, float* dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

// head: identical math to the fused path's head, fp32 or bf16 weight
__global__ void g_head(const float* h, int S, int T, int d, float eps, const float* gfin, const void* w, int wdtype,
                       int n_out, float* wp) {
  __shared__ float red[16];
  extern __shared__ float xm[];
  const int b = blockIdx.x;
  for (int n = threadIdx.x; n < d; n += blockDim.x) xm[n] = 0.f;
  for (int t = 0; t < T; ++t) {
    const float* hr = h + ((int64_t)b * S + t) * d;
    float ss = 0.f;
    for (int n = threadIdx.x; n < d; n += blockDim.x) ss += hr[n] * hr[n];
    ss = block_sum(ss, red);
    const float r = 1.0f / sqrtf(ss / (float)d + eps);
    for (int n = threadIdx.x; n < d; n += blockDim.x) xm[n] += hr[n] * r * gfin[n];
  }
  __syncthreads();
  for (int o = threadIdx.x; o < n_out; o += blockDim.x) {
    float acc = 0.f;
    for (int n = 0; n < d; ++n) acc += xm[n] * ld(w, wdtype, (int64_t)o * d + n);
    wp[(int64_t)b * n_out + o] = acc / (float)T;
  }
}

static inline unsigned nblk(int64_t n, int bs) { return (unsigned)((n + bs - 1) / bs); }

hipError_t generic_tick(const GenericWeights* L, const float* final_norm, const void* head_w, const QueryHead& qhead,
                        int wdt,
                        const void* tokens, const CacheView& cv0, const TickParams& tp, const Dims& dm,
                        const GenericWorkspace& ws, float* waypoints, float* hidden, hipStream_t s) {
  const int M = tp.M, d = dm.d, A = dm.A, F = dm.F;
  hipLaunchKernelGGL(g_embed, dim3(M), dim3(128), 0, s, tokens, wdt, tp, dm, ws);
  for (int l = 0; l < dm.n_layers; ++l) {
    CacheView cv = cv0;
    cv.layer = l;
    hipLaunchKernelGGL(g_norm, dim3(M), dim3(256), 0, s, (const float*)ws.h, L[l].attn_norm, ws.x, d, dm.eps);
    hipLaunchKernelGGL(g_linear, dim3(nblk((int64_t)M * A, 256)), dim3(256), 0, s, (const float*)ws.x, L[l].wq, wdt,
                       ws.q, M, A, d, 0);
    hipLaunchKernelGGL(g_linear, dim3(nblk((int64_t)M * A, 256)), dim3(256), 0, s, (const float*)ws.x, L[l].wk, wdt,
                       ws.k, M, A, d, 0);
    hipLaunchKernelGGL(g_linear, dim3(nblk((int64_t)M * A, 256)), dim3(256), 0, s, (const float*)ws.x, L[l].wv, wdt,
                       ws.v, M, A, d, 0);
    hipLaunchKernelGGL(g_rope, dim3(nblk((int64_t)M * dm.H * (dm.Dh / 2), 256)), dim3(256), 0, s, ws.q, ws.k,
                       (const float*)ws.rope, M, dm.H, dm.Dh);
    hipLaunchKernelGGL(g_attention, dim3(nblk((int64_t)M * dm.H, 64)), dim3(64), 0, s, cv, tp, (const float*)ws.q,
                       (const float*)ws.k, (const float*)ws.v, ws.attn, dm.H, dm.Dh);
    hipLaunchKernelGGL(g_linear, dim3(nblk((int64_t)M * d, 256)), dim3(256), 0, s, (const float*)ws.attn, L[l].wo,
                       wdt, ws.h, M, d, A, 1);
    hipLaunchKernelGGL(g_norm, dim3(M), dim3(256), 0, s, (const float*)ws.h, L[l].ffn_norm, ws.x, d, dm.eps);
    hipLaunchKernelGGL(g_linear, dim3(nblk((int64_t)M * F, 256)), dim3(256), 0, s, (const float*)ws.x, L[l].wg, wdt,
                       ws.g, M, F, d, 0);
    hipLaunchKernelGGL(g_linear, dim3(nblk((int64_t)M * F, 256)), dim3(256), 0, s, (const float*)ws.x, L[l].wu, wdt,
                       ws.u, M, F, d, 0);
    hipLaunchKernelGGL(g_swiglu, dim3(nblk((int64_t)M * F, 256)), dim3(256), 0, s, ws.g, (const float*)ws.u,
                       (int64_t)M * F);
    hipLaunchKernelGGL(g_linear, dim3(nblk((int64_t)M * d, 256)), dim3(256), 0, s, (const float*)ws.g, L[l].wd, wdt,
                       ws.h, M, d, F, 1);
    if (hidden)
      hipLaunchKernelGGL(g_copy, dim3(nblk((int64_t)M * d, 256)), dim3(256), 0, s, (const float*)ws.h,
                         hidden + (int64_t)l * M * d, (int64_t)M * d);
  }
  if (dm.head_kind == 1) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_query_head((const float*)ws.h, tp, dm, final_norm, qhead, waypoints, s);
  }
  hipLaunchKernelGGL(g_head, dim3(tp.B), dim3(256), d * sizeof(float), s, (const float*)ws.h, tp.S, tp.T, d, dm.eps,
                     final_norm, head_w, wdt, dm.n_out, waypoints);
  return hipGetLastError();
}

}  // namespace fsx
