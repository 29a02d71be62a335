// Kernels of the bf16 expert tick on gfx950 (Sec. 3.1, Eq. (1); Sec. 3.3).
//
// One tick, per layer:
//   qkv   : x = RMSNorm(h) (bf16) times the packed [3A][d] projection on MFMA; epilogue applies the
//           rotary rotation to q and k and folds 1/sqrt(Dh) * log2(e) into q.
//   attn  : split-K ("flash-decode") joint attention.  A work item is (agent, head, chunk of cached
//           rows, tile of 16 queries); the expert's own keys/values form one extra chunk per agent, so
//           Eq. (1)'s single softmax over [cache ; own rows] is the log-sum-exp merge of the items.
//   comb  : merges the items of each (agent, head) and writes the attention output (bf16).
//   o     : output projection, split-K partial sums.
//   norm  : h += sum of partials; x = RMSNorm(h) * gain (bf16) for the next projection.
//   gu    : gate/up projection on MFMA with SwiGLU in the epilogue.
//   down  : down projection, split-K partials; then norm again with the next layer's gain.
// The head pools the first T tokens after a final RMSNorm and applies a d -> n_out map.

#include <algorithm>

#include "attn_device.h"
#include "common.h"
#include "kernels.h"

namespace fsx {

// =====================================================================================================
// Weight packing.  A [N][K] bf16 matrix (nn.Linear layout) becomes N/16 x K/32 blocks of 1 KiB; block
// (nt, kb) sits at element offset (nt*K/32 + kb)*512 and its 16-byte slot l (l = 0..63) holds
// W[row(nt*16 + l%16)][kb*32 + 8*(l/16) + j], j = 0..7 -- exactly the B operand of a 16x16x32 MFMA for
// output columns nt*16.. and k = kb*32.., so one wave reads a block with one fully coalesced 1 KiB load.
// row() pairs rows for fused epilogues:
//   PACK_ROPE_PAIRS  : within each head of width Dh, tile tau holds channels [8tau, 8tau+8) in columns
//                      0..7 and [Dh/2 + 8tau, ...) in columns 8..15, so rotary partners are lanes l, l^8.
//   PACK_SWIGLU_PAIRS: tile tau holds gate rows [8tau, 8tau+8) (from a) in columns 0..7 and the same up
//                      rows (from b) in columns 8..15.
// When the projection reads an RMSNorm output, the norm's gain is folded into the packed weights
// (x*r*g) W^T = r * (x (W diag(g))^T), so kernels feed bf16(x) and scale each output row by r.
// =====================================================================================================
__global__ void k_pack(const uint16_t* __restrict__ a, const uint16_t* __restrict__ b, int N, int K, int kind,
                       int param, const float* __restrict__ gain, uint4* __restrict__ dst) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int KB = K / 32;
  const int64_t total = (int64_t)(N / 16) * KB * 64;
  if (i >= total) return;
  const int l = (int)(i & 63);
  const int64_t blk = i >> 6;
  const int kb = (int)(blk % KB);
  const int nt = (int)(blk / KB);
  const int n = nt * 16 + (l & 15);
  const int kcol = kb * 32 + 8 * (l >> 4);
  const uint16_t* src = a;
  int64_t row = n;
  if (kind == PACK_ROPE_PAIRS) {
    const int Dh = param, half = Dh / 2;
    const int head = n / Dh, p = n % Dh, tau = p / 16, c = p % 16;
    row = (int64_t)head * Dh + (c < 8 ? 8 * tau + c : half + 8 * tau + (c - 8));
  } else if (kind == PACK_SWIGLU_PAIRS) {
    const int tau = n / 16, c = n % 16;
    row = 8 * tau + (c & 7);
    src = c < 8 ? a : b;
  }
  uint4 v = *reinterpret_cast<const uint4*>(src + row * K + kcol);
  if (gain) {  // fold the RMSNorm gain of the input channels into the weight: W'[n][k] = W[n][k] * g[k]
    uint32_t* w = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float lo = bf16_to_f32((uint16_t)(w[j] & 0xffffu)) * gain[kcol + 2 * j];
      const float hi = bf16_to_f32((uint16_t)(w[j] >> 16)) * gain[kcol + 2 * j + 1];
      w[j] = pack_bf16x2(lo, hi);
    }
  }
  dst[i] = v;
}

hipError_t launch_pack(const uint16_t* a, const uint16_t* b, int N, int K, int kind, int param, const float* gain,
                       void* dst, hipStream_t s) {
  const int64_t total = (int64_t)(N / 16) * (K / 32) * 64;
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)blocks), dim3(256), 0, s, a, b, N, K, kind, param, gain, (uint4*)dst);
  return hipGetLastError();
}

// =====================================================================================================
// Embed: h = tokens (fp32), x = bf16(h / rms(h)), rotary table cos/sin(p * base^(-2j/Dh)) in fp64.
// One workgroup per token row.
// =====================================================================================================
__global__ __launch_bounds__(256) void k_embed(const void* __restrict__ tokens, int tok_dtype,
                                               const float* __restrict__ g0, TickParams tp, Dims dm,
                                               Workspace ws) {
  __shared__ float red[16];
  const int m = blockIdx.x;
  const int b = m / tp.S, t = m % tp.S;
  const int d = dm.d;
  float ss = 0.f;
  for (int n = threadIdx.x; n < d; n += blockDim.x) {
    const int64_t idx = (int64_t)m * d + n;
    const float v = tok_dtype == FSX_BF16 ? bf16_to_f32(((const uint16_t*)tokens)[idx]) : ((const float*)tokens)[idx];
    ws.h[idx] = v;
    ss += v * v;
  }
  ss = block_sum(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)d + dm.eps);
  for (int n = threadIdx.x; n < d; n += blockDim.x) {
    const int64_t idx = (int64_t)m * d + n;
    ws.xb[idx] = f32_to_bf16(ws.h[idx] * r);  // the gain is folded into the packed weights
  }
  const int half = dm.Dh / 2;
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    double cs = 1.0, sn = 0.0;
    if (dm.rope_base > 0.f) {
      const double theta = pow((double)dm.rope_base, -2.0 * (double)j / (double)dm.Dh);
      const double ang = (double)(tp.pos[b] + t) * theta;
      cs = cos(ang);
      sn = sin(ang);
    }
    ws.rope[((int64_t)m * half + j) * 2 + 0] = (float)cs;
    ws.rope[((int64_t)m * half + j) * 2 + 1] = (float)sn;
  }
}

hipError_t launch_embed(const void* tokens, int tok_dtype, const float* g0, const TickParams& tp, const Dims& dm,
                        const Workspace& ws, hipStream_t s) {
  hipLaunchKernelGGL(k_embed, dim3(tp.M), dim3(256), 0, s, tokens, tok_dtype, g0, tp, dm, ws);
  return hipGetLastError();
}

// =====================================================================================================
// Projection GEMM: y[m][n] = sum_k x[m][k] W[n][k], x bf16 [M][K], W packed (above).
// Workgroup = 4 waves on one 16-column tile and one split-K range; the waves interleave its k-blocks,
// then reduce their accumulators through LDS.  Each lane streams one 16-byte weight slot per k-block
// (1 KiB coalesced per wave) and multiplies it by up to MT 16-row tiles of x.
// =====================================================================================================
enum { EPI_QKV = 0, EPI_SWIGLU = 1, EPI_PARTIAL = 2 };

struct GemmArgs {
  const uint16_t* x;
  int ldx;
  const uint4* w;
  int M, K, N, ksplit;
  float* out_f;      // QKV: q [M][A]; PARTIAL: [ksplit][M][N]
  uint16_t* out_k;   // QKV
  uint16_t* out_v;   // QKV
  uint16_t* out_z;   // SWIGLU: [M][N/2]
  const float* rope; // [M][Dh/2][2]
  int A, Dh;
  float q_scale;
  // optional RMSNorm scale of each row [M], applied to the products (wide rows: x then holds the unscaled residual
  // in bf16; the gain is folded into the weights)
  const float* rscale;
};

template <int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, f32x4 s, int row0, int nt, int ks, int c, int grp) {
  const int n = nt * 16 + c;
  if constexpr (EPI == EPI_PARTIAL) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = row0 + 4 * grp + i;
      if (row < g.M) g.out_f[((int64_t)ks * g.M + row) * g.N + n] = s[i];
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float up = xor8(s[i]);
      const int row = row0 + 4 * grp + i;
      if (c < 8 && row < g.M) {
        const float gt = s[i];
        const float zz = gt / (1.0f + expf(-gt)) * up;
        g.out_z[(int64_t)row * (g.N / 2) + nt * 8 + c] = f32_to_bf16(zz);
      }
    }
  } else {
    const int A = g.A, Dh = g.Dh, half = Dh / 2;
    const int sec = n / A;  // 0 = q, 1 = k, 2 = v (uniform across the tile)
    const int nl = n - sec * A;
    if (sec == 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = row0 + 4 * grp + i;
        if (row < g.M) g.out_v[(int64_t)row * A + nl] = f32_to_bf16(s[i]);
      }
    } else {
      const int head = nl / Dh, p = nl % Dh;
      const int j = 8 * (p / 16) + (c & 7);
      const int dch = c < 8 ? j : half + j;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float other = xor8(s[i]);
        const int row = row0 + 4 * grp + i;
        const int rrow = row < g.M ? row : 0;
        const float cs = g.rope[((int64_t)rrow * half + j) * 2 + 0];
        const float sn = g.rope[((int64_t)rrow * half + j) * 2 + 1];
        const float r = c < 8 ? s[i] * cs - other * sn : s[i] * cs + other * sn;
        if (row < g.M) {
          const int64_t o = (int64_t)row * A + head * Dh + dch;
          if (sec == 0)
            g.out_f[o] = r * g.q_scale;
          else
            g.out_k[o] = f32_to_bf16(r);
        }
      }
    }
  }
}

template <int MT, int EPI>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g) {
  __shared__ f32x4 red[4][MT][WAVE];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = lane & 15, grp = lane >> 4;
  const int n_tiles = g.N / 16;
  const int nt = blockIdx.x % n_tiles, ks = blockIdx.x / n_tiles;
  const int KB = g.K / 32;
  const int kbs = KB / g.ksplit;
  const int kb0 = ks * kbs, kb1 = kb0 + kbs;
  const uint4* __restrict__ wt = g.w + (int64_t)nt * KB * WAVE + lane;
  const int n_mt = (g.M + 15) / 16;
  for (int mg = 0; mg < n_mt; mg += MT) {
    f32x4 acc[MT];
    const uint16_t* xr[MT];
    bool ok[MT];
    float rsc[MT][4];  // row scales of this lane's epilogue rows, loaded before the weight stream
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int row = (mg + mt) * 16 + c;
      ok[mt] = row < g.M;
      xr[mt] = g.x + (int64_t)(ok[mt] ? row : 0) * g.ldx + 8 * grp;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int er = (mg + mt) * 16 + 4 * grp + i;
        rsc[mt][i] = EPI != EPI_PARTIAL && g.rscale && er < g.M ? g.rscale[er] : 1.f;
      }
    }
    // Batches of U k-blocks of this wave: every weight block and x operand of the batch is loaded before the first
    // MFMA, so U KiB of weights per wave are in flight (one at a time leaves the stream latency-bound).
    constexpr int U = MT <= 1 ? 8 : (MT <= 2 ? 6 : (MT <= 4 ? 4 : 2));
    int kb = kb0 + wave;
    for (; kb + 4 * (U - 1) < kb1; kb += 4 * U) {
      uint4 wv[U], xv[U][MT];
#pragma unroll
      for (int u = 0; u < U; ++u) wv[u] = ld_global(wt + (int64_t)(kb + 4 * u) * WAVE);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          xv[u][mt] = ok[mt] ? *reinterpret_cast<const uint4*>(xr[mt] + (kb + 4 * u) * 32) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = mfma_bf16(xv[u][mt], wv[u], acc[mt]);
    }
    if (kb < kb1) {
      // the last, partial batch: its k-blocks loaded together too (the missing ones as zeros), so a short split-K
      // range costs one load latency instead of one per k-block
      uint4 wv[U], xv[U][MT];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = kb + 4 * u < kb1;
        wv[u] = in ? ld_global(wt + (int64_t)(kb + 4 * u) * WAVE) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          xv[u][mt] = in && ok[mt] ? *reinterpret_cast<const uint4*>(xr[mt] + (kb + 4 * u) * 32) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (kb + 4 * u < kb1)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[mt] = mfma_bf16(xv[u][mt], wv[u], acc[mt]);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) red[wave][mt][lane] = acc[mt];
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (mt % 4 != wave) continue;
      f32x4 s = red[0][mt][lane] + red[1][mt][lane] + red[2][mt][lane] + red[3][mt][lane];
#pragma unroll
      for (int i = 0; i < 4; ++i) s[i] *= rsc[mt][i];
      gemm_epilogue<EPI>(g, s, (mg + mt) * 16, nt, ks, c, grp);
    }
    __syncthreads();
  }
}

// Projection of batched rows: CT column tiles per workgroup, so each row operand loaded from L2 serves CT tiles (with
// one tile per workgroup the rows' bytes were MT times the weights' for MT row tiles).  The 4 waves split K as in
// k_gemm; wave w holds U batches of CT weight blocks and MT row operands, then runs CT x MT MFMA chains.
template <int MT, int CT, int EPI>
__global__ __launch_bounds__(256) void k_gemm_ct(GemmArgs g) {
  __shared__ f32x4 red[4][CT][MT][WAVE];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = lane & 15, grp = lane >> 4;
  const int n_groups = g.N / (16 * CT);
  const int ng = blockIdx.x % n_groups, ks = blockIdx.x / n_groups;
  const int KB = g.K / 32;
  const int kbs = KB / g.ksplit;
  const int kb0 = ks * kbs, kb1 = kb0 + kbs;
  const uint4* __restrict__ wt = g.w + (int64_t)ng * CT * KB * WAVE + lane;  // tile ct at wt + ct * KB * WAVE
  const int n_mt = (g.M + 15) / 16;
  for (int mg = 0; mg < n_mt; mg += MT) {
    f32x4 acc[CT][MT];
    const uint16_t* xr[MT];
    bool ok[MT];
    float rsc[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) acc[ct][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int row = (mg + mt) * 16 + c;
      ok[mt] = row < g.M;
      xr[mt] = g.x + (int64_t)(ok[mt] ? row : 0) * g.ldx + 8 * grp;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int er = (mg + mt) * 16 + 4 * grp + i;
        rsc[mt][i] = EPI != EPI_PARTIAL && g.rscale && er < g.M ? g.rscale[er] : 1.f;
      }
    }
    constexpr int U = 2;
    int kb = kb0 + wave;
    for (; kb + 4 * (U - 1) < kb1; kb += 4 * U) {
      uint4 wv[U][CT], xv[U][MT];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) wv[u][ct] = ld_global(wt + ((int64_t)ct * KB + kb + 4 * u) * WAVE);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          xv[u][mt] = ok[mt] ? *reinterpret_cast<const uint4*>(xr[mt] + (kb + 4 * u) * 32) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[ct][mt] = mfma_bf16(xv[u][mt], wv[u][ct], acc[ct][mt]);
    }
    if (kb < kb1) {  // the last, partial batch, loaded together as in k_gemm
      uint4 wv[U][CT], xv[U][MT];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = kb + 4 * u < kb1;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
          wv[u][ct] = in ? ld_global(wt + ((int64_t)ct * KB + kb + 4 * u) * WAVE) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          xv[u][mt] = in && ok[mt] ? *reinterpret_cast<const uint4*>(xr[mt] + (kb + 4 * u) * 32) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (kb + 4 * u < kb1)
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[ct][mt] = mfma_bf16(xv[u][mt], wv[u][ct], acc[ct][mt]);
    }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) red[wave][ct][mt][lane] = acc[ct][mt];
    __syncthreads();
#pragma unroll
    for (int p = 0; p < CT * MT; ++p) {
      if (p % 4 != wave) continue;
      const int ct = p / MT, mt = p % MT;
      f32x4 sm = red[0][ct][mt][lane] + red[1][ct][mt][lane] + red[2][ct][mt][lane] + red[3][ct][mt][lane];
#pragma unroll
      for (int i = 0; i < 4; ++i) sm[i] *= rsc[mt][i];
      gemm_epilogue<EPI>(g, sm, (mg + mt) * 16, ng * CT + ct, ks, c, grp);
    }
    __syncthreads();
  }
}

template <int EPI>
static hipError_t gemm_dispatch(const GemmArgs& g, hipStream_t s) {
  const int n_mt = (g.M + 15) / 16;
  const int groups = (n_mt + 7) / 8;
  const int mt = (n_mt + groups - 1) / groups;
  // several column tiles per workgroup when the rows span more than one tile and the grid still fills the chip
  const int tiles = g.N / 16;
  auto fills = [&](int ct) { return tiles % ct == 0 && (tiles / ct) * g.ksplit >= 256; };
  const dim3 block(256);
  if (mt >= 2 && mt <= 4 && fills(4)) {
    const dim3 grid((unsigned)((tiles / 4) * g.ksplit));
    switch (mt) {
      case 2: hipLaunchKernelGGL((k_gemm_ct<2, 4, EPI>), grid, block, 0, s, g); break;
      case 3: hipLaunchKernelGGL((k_gemm_ct<3, 4, EPI>), grid, block, 0, s, g); break;
      default: hipLaunchKernelGGL((k_gemm_ct<4, 4, EPI>), grid, block, 0, s, g); break;
    }
    return hipGetLastError();
  }
  if (mt >= 2 && fills(2)) {
    const dim3 grid((unsigned)((tiles / 2) * g.ksplit));
    switch (mt) {
      case 2: hipLaunchKernelGGL((k_gemm_ct<2, 2, EPI>), grid, block, 0, s, g); break;
      case 3: hipLaunchKernelGGL((k_gemm_ct<3, 2, EPI>), grid, block, 0, s, g); break;
      case 4: hipLaunchKernelGGL((k_gemm_ct<4, 2, EPI>), grid, block, 0, s, g); break;
      case 5: hipLaunchKernelGGL((k_gemm_ct<5, 2, EPI>), grid, block, 0, s, g); break;
      case 6: hipLaunchKernelGGL((k_gemm_ct<6, 2, EPI>), grid, block, 0, s, g); break;
      case 7: hipLaunchKernelGGL((k_gemm_ct<7, 2, EPI>), grid, block, 0, s, g); break;
      default: hipLaunchKernelGGL((k_gemm_ct<8, 2, EPI>), grid, block, 0, s, g); break;
    }
    return hipGetLastError();
  }
  const dim3 grid((unsigned)(tiles * g.ksplit));
  switch (mt) {
    case 1: hipLaunchKernelGGL((k_gemm<1, EPI>), grid, block, 0, s, g); break;
    case 2: hipLaunchKernelGGL((k_gemm<2, EPI>), grid, block, 0, s, g); break;
    case 3: hipLaunchKernelGGL((k_gemm<3, EPI>), grid, block, 0, s, g); break;
    case 4: hipLaunchKernelGGL((k_gemm<4, EPI>), grid, block, 0, s, g); break;
    case 5: hipLaunchKernelGGL((k_gemm<5, EPI>), grid, block, 0, s, g); break;
    case 6: hipLaunchKernelGGL((k_gemm<6, EPI>), grid, block, 0, s, g); break;
    case 7: hipLaunchKernelGGL((k_gemm<7, EPI>), grid, block, 0, s, g); break;
    default: hipLaunchKernelGGL((k_gemm<8, EPI>), grid, block, 0, s, g); break;
  }
  return hipGetLastError();
}

// After a reduction of wide rows xb holds the unscaled residual and ws.rs each row's RMSNorm scale: the
// projection applies the scales to its products.
static void row_scale_from_chunks(GemmArgs& g, const Dims& dm, const Workspace& ws, bool after_reduction) {
  if (after_reduction && wide_rows(dm)) g.rscale = ws.rs;
}

hipError_t launch_gemm_qkv(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                           hipStream_t s, bool after_reduction) {
  GemmArgs g{};
  g.x = ws.xb; g.ldx = dm.d; g.w = w.wqkv; g.M = tp.M; g.K = dm.d; g.N = 3 * dm.A; g.ksplit = 1;
  row_scale_from_chunks(g, dm, ws, after_reduction);
  g.out_f = ws.q; g.out_k = ws.kself; g.out_v = ws.vself; g.rope = ws.rope; g.A = dm.A; g.Dh = dm.Dh;
  g.q_scale = LOG2E / sqrtf((float)dm.Dh);
  return gemm_dispatch<EPI_QKV>(g, s);
}

hipError_t launch_gemm_o(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                         int ksplit, hipStream_t s) {
  GemmArgs g{};
  g.x = ws.attn; g.ldx = dm.A; g.w = w.wo; g.M = tp.M; g.K = dm.A; g.N = dm.d; g.ksplit = ksplit;
  g.out_f = ws.part;
  return gemm_dispatch<EPI_PARTIAL>(g, s);
}

hipError_t launch_gemm_gu(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                          hipStream_t s) {
  GemmArgs g{};
  g.x = ws.xb; g.ldx = dm.d; g.w = w.wgu; g.M = tp.M; g.K = dm.d; g.N = 2 * dm.F; g.ksplit = 1;
  g.out_z = ws.z;
  row_scale_from_chunks(g, dm, ws, true);
  return gemm_dispatch<EPI_SWIGLU>(g, s);
}

hipError_t launch_gemm_down(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                            int ksplit, hipStream_t s) {
  GemmArgs g{};
  g.x = ws.z; g.ldx = dm.F; g.w = w.wd; g.M = tp.M; g.K = dm.F; g.N = dm.d; g.ksplit = ksplit;
  g.out_f = ws.part;
  return gemm_dispatch<EPI_PARTIAL>(g, s);
}

// =====================================================================================================
// Split-K joint attention (Eq. (1)): one wave = one work item (see attn_device.h); k_combine merges the
// items of each (agent, head, query tile).
// =====================================================================================================
struct AttnArgs {
  CacheView cv;
  const float* q;
  const uint16_t* kself;
  const uint16_t* vself;
  float* att_o;
  float* att_ml;
  uint16_t* attn_out;  // [M][A] bf16 (combine output)
  int H, Dh, A;
  int causal;          // the own rows are masked causally (new token t sees own rows 0..t)
  int write_rows;      // combine launch: also store the new rows (kself/vself) into the cache rings (cv)
};

template <int KT>
__global__ __launch_bounds__(256) void k_attention(AttnArgs a, TickParams tp) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int item = blockIdx.x * (blockDim.x >> 6) + wave;
  if (item >= tp.n_items) return;
  const int tt = item % tp.n_tt;
  const int rest = item / tp.n_tt;
  const int h = rest % a.H;
  const int cs = rest / a.H;
  int b = 0;
  while (b + 1 < tp.B && tp.chunk_prefix[b + 1] <= cs) ++b;
  const int cidx = cs - tp.chunk_prefix[b];
  const int nch = tp.chunk_prefix[b + 1] - tp.chunk_prefix[b] - 1;
  const int grp = lane >> 4;
  const int t = tt * 16 + (lane & 15);
  const bool tv = t < tp.S;
  const int64_t qrow = ((int64_t)b * tp.S + (tv ? t : 0)) * a.A + (int64_t)h * a.Dh;
  float* out_o = a.att_o + (int64_t)item * 16 * a.Dh;
  float* out_ml = a.att_ml + (int64_t)item * 32;
  uint4 qf[4];
  if (cidx == nch) {  // the expert's own rows (bf16)
    load_q_frag<0, false>(a.q, qrow, tv, grp, qf);
    const int64_t off = ((int64_t)b * tp.S * a.A + (int64_t)h * a.Dh) * 2;
    attn_rows<0, false, false, false>((const char*)a.kself + off, (const char*)a.vself + off, (int64_t)a.A * 2, 0, 0, 0, tp.S, qf,
                        1.f, 1.f, lane, out_o, out_ml, a.Dh, a.causal ? tt * 16 : 1 << 30);
  } else {
    const int i0 = cidx * tp.chunk_rows;
    const int i1 = min(i0 + tp.chunk_rows, tp.len[b]);
    constexpr int ES = KT == 0 ? 2 : 1;
    // ring slot 0 of (agent, layer, head); slots are a.cv.rs elements apart
    const int64_t off = cache_head_base(a.cv, b, a.cv.layer, h) * ES;
    float ks = 1.f, vs = 1.f;
    if (KT == 1) {
      const int64_t si = cache_scale_index(a.cv, b, a.cv.layer, h);
      ks = a.cv.k_scale[si];
      vs = a.cv.v_scale[si];
    }
    load_q_frag<KT, false>(a.q, qrow, tv, grp, qf);
    attn_rows<KT, true, false, false>((const char*)a.cv.k + off, (const char*)a.cv.v + off, a.cv.rs * ES, tp.start[b],
                        a.cv.cap, i0, i1, qf, ks, vs, lane, out_o, out_ml, a.Dh);
  }
}

hipError_t launch_attention(const CacheView& cv, const TickParams& tp, const Dims& dm, const Workspace& ws,
                            int waves_per_wg, hipStream_t s, bool causal) {
  AttnArgs a{};
  a.cv = cv; a.q = ws.q; a.kself = ws.kself; a.vself = ws.vself; a.att_o = ws.att_o; a.att_ml = ws.att_ml;
  a.H = dm.H; a.Dh = dm.Dh; a.A = dm.A; a.causal = causal ? 1 : 0;
  const dim3 grid((unsigned)((tp.n_items + waves_per_wg - 1) / waves_per_wg)), block(64 * waves_per_wg);
  if (cv.dtype == FSX_FP8_E4M3)
    hipLaunchKernelGGL(k_attention<1>, grid, block, 0, s, a, tp);
  else
    hipLaunchKernelGGL(k_attention<0>, grid, block, 0, s, a, tp);
  return hipGetLastError();
}

// Log-sum-exp merge of the work items of one (agent, head, query tile), in item order.
__device__ __forceinline__ void write_row_chunk(const CacheView& cv, const uint16_t* ks, const uint16_t* vs,
                                                const TickParams& tp, int64_t i);

// Workgroups past the B * H * n_tt merges (when a.write_rows is set) store the layer's new rows into the cache.
__global__ __launch_bounds__(256) void k_combine(AttnArgs a, TickParams tp) {
  const int n_merge = tp.B * a.H * tp.n_tt;
  if ((int)blockIdx.x >= n_merge) {
    write_row_chunk(a.cv, a.kself, a.vself, tp, (int64_t)(blockIdx.x - n_merge) * blockDim.x + threadIdx.x);
    return;
  }
  const int tt = blockIdx.x % tp.n_tt;
  const int rest = blockIdx.x / tp.n_tt;
  const int h = rest % a.H;
  const int b = rest / a.H;
  const int first = tp.chunk_prefix[b], nslot = tp.chunk_prefix[b + 1] - first;
  const int t = threadIdx.x >> 4, d0 = (threadIdx.x & 15) * 8;
  float M = -INFINITY;
  for (int sl = 0; sl < nslot; ++sl) {
    const int64_t item = ((int64_t)(first + sl) * a.H + h) * tp.n_tt + tt;
    M = fmaxf(M, a.att_ml[item * 32 + t * 2]);
  }
  float L = 0.f, acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.f;
  for (int sl = 0; sl < nslot; ++sl) {
    const int64_t item = ((int64_t)(first + sl) * a.H + h) * tp.n_tt + tt;
    const float w = exp2f(a.att_ml[item * 32 + t * 2] - M);
    L += a.att_ml[item * 32 + t * 2 + 1] * w;
    const float4* po = reinterpret_cast<const float4*>(a.att_o + (item * 16 + t) * a.Dh + d0);
    const float4 x0 = po[0], x1 = po[1];
    acc[0] += x0.x * w; acc[1] += x0.y * w; acc[2] += x0.z * w; acc[3] += x0.w * w;
    acc[4] += x1.x * w; acc[5] += x1.y * w; acc[6] += x1.z * w; acc[7] += x1.w * w;
  }
  const int tok = tt * 16 + t;
  if (tok < tp.S) {
    const float inv = 1.0f / L;
    const uint4 out = make_uint4(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                                 pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv));
    *reinterpret_cast<uint4*>(a.attn_out + ((int64_t)b * tp.S + tok) * a.A + (int64_t)h * a.Dh + d0) = out;
  }
}

hipError_t launch_combine(const TickParams& tp, const Dims& dm, const Workspace& ws, hipStream_t s,
                          const CacheView* rows_into) {
  AttnArgs a{};
  a.att_o = ws.att_o; a.att_ml = ws.att_ml; a.attn_out = ws.attn; a.H = dm.H; a.Dh = dm.Dh; a.A = dm.A;
  int64_t blocks = (int64_t)tp.B * dm.H * tp.n_tt;
  if (rows_into) {
    a.cv = *rows_into;
    a.kself = ws.kself;
    a.vself = ws.vself;
    a.write_rows = 1;
    blocks += ((int64_t)tp.B * tp.S * rows_into->H * (rows_into->Dh / 8) + 255) / 256;
  }
  hipLaunchKernelGGL(k_combine, dim3((unsigned)blocks), dim3(256), 0, s, a, tp);
  return hipGetLastError();
}

// =====================================================================================================
// h += sum of split-K partials (fixed order), optional copy to the per-layer hidden output, then
// x = bf16(h / rms(h)) for the next projection (whose packed weights carry the norm gain).  One workgroup
// per token row.
// =====================================================================================================
__global__ __launch_bounds__(256) void k_reduce_norm(float* __restrict__ h, const float* __restrict__ part,
                                                     uint16_t* __restrict__ xb, int M, int d, int ksplit,
                                                     const float* __restrict__ gain, float eps,
                                                     float* __restrict__ hidden) {
  __shared__ float red[16];
  const int m = blockIdx.x;
  float ss = 0.f;
  for (int n = threadIdx.x; n < d; n += blockDim.x) {
    const int64_t idx = (int64_t)m * d + n;
    float acc = 0.f;
    for (int s = 0; s < ksplit; ++s) acc += part[((int64_t)s * M + m) * d + n];
    const float v = h[idx] + acc;
    h[idx] = v;
    if (hidden) hidden[idx] = v;
    ss += v * v;
  }
  ss = block_sum(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  for (int n = threadIdx.x; n < d; n += blockDim.x) {
    const int64_t idx = (int64_t)m * d + n;
    xb[idx] = f32_to_bf16(h[idx] * r);  // the gain is folded into the packed weights
  }
}

// Wide rows (the backbone's d = 4096 over a handful of tokens): one workgroup per row leaves the partial sums'
// loads latency-bound on a few CUs, so the rows are cut into 512-column chunks, one workgroup each: h += sum of the
// partials, xb = bf16(h) unscaled, and the chunk's sum of squares to ss[m][chunk]; the last chunk of the row forms
// the row's RMSNorm scale, which the next projection applies to its products, so no launch forms the normalised
// input.
__global__ __launch_bounds__(RN_CHUNK / 4) void k_reduce_chunks(float* __restrict__ h, const float* __restrict__ part,
                                                                int M, int d, int ksplit, float* __restrict__ ss,
                                                                uint16_t* __restrict__ xb, float* __restrict__ hidden,
                                                                float* __restrict__ rs, uint32_t* __restrict__ rcnt,
                                                                float eps) {
  __shared__ float red[16];
  const int nch = d / RN_CHUNK, m = blockIdx.x / nch, ch = blockIdx.x % nch;
  // thread t: the 4 columns ch * RN_CHUNK + 4t .. + 3, 16-byte loads (every partial's load issued before any add)
  const int64_t idx = (int64_t)m * d + ch * RN_CHUNK + 4 * threadIdx.x;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = 0; s0 < ksplit; s0 += 8) {
    float4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      v[j] = s0 + j < ksplit ? *reinterpret_cast<const float4*>(part + (int64_t)(s0 + j) * M * d + idx)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      acc.x += v[j].x;
      acc.y += v[j].y;
      acc.z += v[j].z;
      acc.w += v[j].w;
    }
  }
  const float4 h0 = *reinterpret_cast<const float4*>(h + idx);
  const float4 val = make_float4(h0.x + acc.x, h0.y + acc.y, h0.z + acc.z, h0.w + acc.w);
  *reinterpret_cast<float4*>(h + idx) = val;
  *reinterpret_cast<uint2*>(xb + idx) = make_uint2(pack_bf16x2(val.x, val.y), pack_bf16x2(val.z, val.w));
  if (hidden) {  // the caller's buffer: 4-byte alignment only
    hidden[idx] = val.x;
    hidden[idx + 1] = val.y;
    hidden[idx + 2] = val.z;
    hidden[idx + 3] = val.w;
  }
  float sq = val.x * val.x + val.y * val.y + val.z * val.z + val.w * val.w;
  sq = block_sum(sq, red);
  // the last chunk of row m to finish adds the chunk sums in chunk order and writes the row's scale; it then resets
  // the row's counter for the next reduction (the next launch).  The sums are device-scope stores completed before
  // the count (no release fence: at device scope that writes back the whole L2) and read with device-scope loads.
  if (threadIdx.x == 0) {
    st_dev_f(ss + (int64_t)m * nch + ch, sq);
    stores_done();
    const uint32_t done = __hip_atomic_fetch_add(rcnt + m, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (done == (uint32_t)(nch - 1)) {
      float tot = 0.f;
      for (int c = 0; c < nch; ++c) tot += ld_dev_f(ss + (int64_t)m * nch + c);
      rs[m] = 1.0f / sqrtf(tot / (float)d + eps);
      __hip_atomic_store(rcnt + m, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

hipError_t launch_reduce_norm(const TickParams& tp, const Dims& dm, const Workspace& ws, int ksplit,
                              const float* gain, float* hidden_layer, hipStream_t s) {
  if (wide_rows(dm)) {
    const int nch = dm.d / RN_CHUNK;
    hipLaunchKernelGGL(k_reduce_chunks, dim3(tp.M * nch), dim3(RN_CHUNK / 4), 0, s, ws.h, (const float*)ws.part, tp.M, dm.d,
                       ksplit, ws.ss, ws.xb, hidden_layer, ws.rs, ws.rcnt, dm.eps);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_reduce_norm, dim3(tp.M), dim3(256), 0, s, ws.h, (const float*)ws.part, ws.xb, tp.M, dm.d,
                     ksplit, gain, dm.eps, hidden_layer);
  return hipGetLastError();
}

// =====================================================================================================
// Waypoint head: mean over the first T tokens of RMSNorm(h) * g_final, then W_head [n_out][d] (no bias).
// One workgroup per agent.  Dynamic LDS: d floats.
// =====================================================================================================
__global__ __launch_bounds__(256) void k_head(const float* __restrict__ h, int S, int T, int d, float eps,
                                              const float* __restrict__ gfin, const void* __restrict__ w,
                                              int wdtype, int n_out, float* __restrict__ wp) {
  extern __shared__ float xm[];
  __shared__ float red[16];
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
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  for (int o = wave; o < n_out; o += nw) {
    float acc = 0.f;
    for (int n = lane; n < d; n += WAVE) {
      const float wv = wdtype == FSX_BF16 ? bf16_to_f32(((const uint16_t*)w)[(int64_t)o * d + n])
                                          : ((const float*)w)[(int64_t)o * d + n];
      acc += xm[n] * wv;
    }
    acc = wave_sum(acc);
    if (lane == 0) wp[(int64_t)b * n_out + o] = acc / (float)T;
  }
}

__global__ __launch_bounds__(256) void k_query_head(const float* __restrict__ h, int S, int T, int d, float eps,
                                                    const float* __restrict__ gfin, QueryHead qh, int nq,
                                                    float* __restrict__ wp) {
  extern __shared__ float qlds[];
  const int b = blockIdx.x;
  query_head_wg([&](int t, int c) { return h[((int64_t)b * S + t) * d + c]; }, T, nq, d, eps, gfin, qh,
                [&](int o, float v) { wp[(int64_t)b * 2 * nq + o] = v; }, qlds);
}

hipError_t launch_query_head(const float* h, const TickParams& tp, const Dims& dm, const float* final_norm,
                             const QueryHead& qh, float* waypoints, hipStream_t s) {
  const int nq = dm.n_out / 2;
  hipLaunchKernelGGL(k_query_head, dim3(tp.B), dim3(256), (size_t)nq * (dm.d + qh.hidden) * sizeof(float), s, h,
                     tp.S, tp.T, dm.d, dm.eps, final_norm, qh, nq, waypoints);
  return hipGetLastError();
}

hipError_t launch_head(const TickParams& tp, const Dims& dm, const Workspace& ws, const float* final_norm,
                       const void* head_w, int head_dtype, float* waypoints, hipStream_t s) {
  hipLaunchKernelGGL(k_head, dim3(tp.B), dim3(256), dm.d * sizeof(float), s, (const float*)ws.h, tp.S, tp.T, dm.d,
                     dm.eps, final_norm, head_w, head_dtype, dm.n_out, waypoints);
  return hipGetLastError();
}

// =====================================================================================================
// Cache append (Sec. 3.3): copy n new rows of every (agent, layer, head) into ring slots
// (first[b] + j) mod cap, bit-exact, 16 bytes per thread.  The rows come in the cache's layout with n slots:
// head-major [B][n_layers][H][n][Dh] into [B][n_layers][H][cap][Dh], or token-major [B][n_layers][n][H][Dh] into
// [B][n_layers][cap][H][Dh].  Either way thread i copies 16-byte chunk i of the source, so reads are coalesced.
// =====================================================================================================
struct AppendArgs {
  const uint4* ks;
  const uint4* vs;
  uint4* kc;
  uint4* vc;
  int64_t cap;
  int64_t row_chunks;  // 16-byte chunks per head row (Dh elements)
  int n_layers, n_heads, n_rows, B, token_major;
  int64_t first[FSX_MAX_BATCH];
};

__global__ __launch_bounds__(256) void k_append(AppendArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)a.B * a.n_layers * a.n_heads * a.n_rows * a.row_chunks;
  if (i >= total) return;
  const int64_t ch = i % a.row_chunks;
  int64_t r = i / a.row_chunks;
  int64_t dst;
  if (a.token_major) {
    const int h = (int)(r % a.n_heads);
    r /= a.n_heads;
    const int j = (int)(r % a.n_rows);
    r /= a.n_rows;  // (b, l)
    const int b = (int)(r / a.n_layers);
    int64_t slot = a.first[b] + j;
    if (slot >= a.cap) slot -= a.cap;
    dst = ((r * a.cap + slot) * a.n_heads + h) * a.row_chunks + ch;
  } else {
    const int j = (int)(r % a.n_rows);
    r /= a.n_rows;  // (b, l, h) slab index
    const int b = (int)(r / ((int64_t)a.n_layers * a.n_heads));
    int64_t slot = a.first[b] + j;
    if (slot >= a.cap) slot -= a.cap;
    dst = (r * a.cap + slot) * a.row_chunks + ch;
  }
  a.kc[dst] = a.ks[i];
  a.vc[dst] = a.vs[i];
}

// Quantising append into an fp8 cache: the rows arrive in bf16 or fp32 and each element is stored as the E4M3 code
// RNE(clamp(x / scale, -448, 448)) with the (agent, layer, head) scale the cache already has.  The encoding follows
// the format's definition step by step (exact in fp32: the quotient is rounded once by the division, the mantissa
// rounding is a rint of an exactly scaled value), so the codes are reproducible bit for bit.
__device__ __forceinline__ uint32_t e4m3_encode(float x, float scale) {
  float y = x / scale;
  if (y != y) return 0x7Fu | (__float_as_uint(y) >> 31 << 7);
  y = fminf(fmaxf(y, -448.0f), 448.0f);
  const uint32_t sign = __float_as_uint(y) >> 31 << 7;
  const float a = fabsf(y);
  uint32_t code;
  if (a < 0.015625f) {  // below the smallest normal 2^-6: subnormal steps of 2^-9
    code = (uint32_t)rintf(a * 512.0f);  // 8 -> the smallest normal, code 0x08
  } else {
    int e;
    const float m = frexpf(a, &e);  // a = m 2^e, m in [0.5, 1)
    uint32_t mant = (uint32_t)rintf((m * 2.0f - 1.0f) * 8.0f);
    int ex = e - 1;
    if (mant == 8) {
      mant = 0;
      ++ex;
    }
    code = ((uint32_t)(ex + 7) << 3) | mant;
  }
  return sign | code;
}

struct QAppendArgs {
  const void* ks;
  const void* vs;
  uint8_t* kc;
  uint8_t* vc;
  const float* kscale;
  const float* vscale;
  int64_t cap;
  int n_layers, n_heads, head_dim, n_rows, B, token_major, src_f32;
  int64_t first[FSX_MAX_BATCH];
};

// Thread i encodes 8 consecutive elements of one head row (8 bytes out).
__global__ __launch_bounds__(256) void k_append_quantize(QAppendArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cpr = a.head_dim / 8;
  const int64_t total = (int64_t)a.B * a.n_layers * a.n_heads * a.n_rows * cpr;
  if (i >= total) return;
  const int ch = (int)(i % cpr);
  int64_t r = i / cpr;
  int b, l, h, j;
  if (a.token_major) {
    h = (int)(r % a.n_heads);
    r /= a.n_heads;
    j = (int)(r % a.n_rows);
    r /= a.n_rows;
    l = (int)(r % a.n_layers);
    b = (int)(r / a.n_layers);
  } else {
    j = (int)(r % a.n_rows);
    r /= a.n_rows;
    h = (int)(r % a.n_heads);
    r /= a.n_heads;
    l = (int)(r % a.n_layers);
    b = (int)(r / a.n_layers);
  }
  int64_t slot = a.first[b] + j;
  if (slot >= a.cap) slot -= a.cap;
  const int64_t lb = ((int64_t)b * a.n_layers + l);
  const int64_t dst = a.token_major ? ((lb * a.cap + slot) * a.n_heads + h) * a.head_dim + 8 * ch
                                    : ((lb * a.n_heads + h) * a.cap + slot) * a.head_dim + 8 * ch;
  const float sk = a.kscale[lb * a.n_heads + h], sv = a.vscale[lb * a.n_heads + h];
  const int64_t src = i * 8;  // the source rows are dense in the same order as i
  float xk[8], xv[8];
  if (a.src_f32) {
    const float4* pk = reinterpret_cast<const float4*>((const float*)a.ks + src);
    const float4* pv = reinterpret_cast<const float4*>((const float*)a.vs + src);
    const float4 k0 = pk[0], k1 = pk[1], v0 = pv[0], v1 = pv[1];
    const float kk[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
    const float vv[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xk[e] = kk[e];
      xv[e] = vv[e];
    }
  } else {
    const uint4 k = *reinterpret_cast<const uint4*>((const uint16_t*)a.ks + src);
    const uint4 v = *reinterpret_cast<const uint4*>((const uint16_t*)a.vs + src);
    const uint32_t kw[4] = {k.x, k.y, k.z, k.w}, vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      xk[2 * e] = __uint_as_float(kw[e] << 16);
      xk[2 * e + 1] = __uint_as_float(kw[e] & 0xFFFF0000u);
      xv[2 * e] = __uint_as_float(vw[e] << 16);
      xv[2 * e + 1] = __uint_as_float(vw[e] & 0xFFFF0000u);
    }
  }
  uint32_t ck[2] = {0, 0}, cv[2] = {0, 0};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    ck[e >> 2] |= e4m3_encode(xk[e], sk) << (8 * (e & 3));
    cv[e >> 2] |= e4m3_encode(xv[e], sv) << (8 * (e & 3));
  }
  *reinterpret_cast<uint2*>(a.kc + dst) = make_uint2(ck[0], ck[1]);
  *reinterpret_cast<uint2*>(a.vc + dst) = make_uint2(cv[0], cv[1]);
}

hipError_t launch_append_quantize(const fsx_cache_desc& c, const void* k_rows, const void* v_rows, int rows_dtype,
                                  int n_rows, const int64_t* first, hipStream_t s) {
  QAppendArgs a{};
  a.ks = k_rows; a.vs = v_rows; a.kc = (uint8_t*)c.k; a.vc = (uint8_t*)c.v; a.kscale = c.k_scale; a.vscale = c.v_scale;
  a.cap = c.capacity; a.n_layers = c.n_layers; a.n_heads = c.n_heads; a.head_dim = c.head_dim; a.n_rows = n_rows;
  a.B = c.batch; a.token_major = (c.layout & FSX_CACHE_TOKEN_MAJOR) != 0; a.src_f32 = rows_dtype == FSX_F32;
  for (int b = 0; b < c.batch; ++b) a.first[b] = first[b];
  const int64_t total = (int64_t)a.B * a.n_layers * a.n_heads * a.n_rows * (a.head_dim / 8);
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(k_append_quantize, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

// The new tokens' rotated keys and values of one layer (kself / vself, bf16 [B*n][H*Dh]) written into that layer's
// ring slots (first[b] + t) mod cap, bf16 copies or fp8 codes against the cache's scales.  Thread i handles 8
// channels of one head row.
// Chunk i (8 elements) of the new rows [B][n][H][Dh] (kself/vself layout, row b * n + t) into ring slot
// (start + len + t) mod capacity of (agent b, layer cv.layer, head h): a bf16 copy, or E4M3 codes with the cache's
// per-(agent, layer, head) scales.  Runs after the attention that read the old rows (a full ring overwrites its
// oldest rows).
__device__ __forceinline__ void write_row_chunk(const CacheView& cv, const uint16_t* ks, const uint16_t* vs,
                                                const TickParams& tp, int64_t i) {
  const int cpr = cv.Dh / 8, A = cv.H * cv.Dh, n = tp.S;
  const int64_t total = (int64_t)tp.B * n * cv.H * cpr;
  if (i >= total) return;
  const int ch = (int)(i % cpr);
  int64_t r = i / cpr;
  const int h = (int)(r % cv.H);
  const int64_t m = r / cv.H;  // token row b * n + t
  const int b = (int)(m / n), t = (int)(m % n);
  int64_t slot = (tp.start[b] + tp.len[b]) % cv.cap + t;
  if (slot >= cv.cap) slot -= cv.cap;
  const int64_t dst = cache_head_base(cv, b, cv.layer, h) + slot * cv.rs + 8 * ch;
  const int64_t src = m * A + (int64_t)h * cv.Dh + 8 * ch;
  const uint4 kv = *reinterpret_cast<const uint4*>(ks + src), vv = *reinterpret_cast<const uint4*>(vs + src);
  if (cv.dtype == FSX_FP8_E4M3) {
    const int64_t si = cache_scale_index(cv, b, cv.layer, h);
    const float sk = cv.k_scale[si], sv = cv.v_scale[si];
    const uint32_t kw[4] = {kv.x, kv.y, kv.z, kv.w}, vw[4] = {vv.x, vv.y, vv.z, vv.w};
    uint32_t ck[2] = {0, 0}, cvw[2] = {0, 0};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t kbits = e & 1 ? kw[e >> 1] & 0xFFFF0000u : kw[e >> 1] << 16;
      const uint32_t vbits = e & 1 ? vw[e >> 1] & 0xFFFF0000u : vw[e >> 1] << 16;
      ck[e >> 2] |= e4m3_encode(__uint_as_float(kbits), sk) << (8 * (e & 3));
      cvw[e >> 2] |= e4m3_encode(__uint_as_float(vbits), sv) << (8 * (e & 3));
    }
    *reinterpret_cast<uint2*>((uint8_t*)cv.k + dst) = make_uint2(ck[0], ck[1]);
    *reinterpret_cast<uint2*>((uint8_t*)cv.v + dst) = make_uint2(cvw[0], cvw[1]);
  } else {
    *reinterpret_cast<uint4*>((uint16_t*)cv.k + dst) = kv;
    *reinterpret_cast<uint4*>((uint16_t*)cv.v + dst) = vv;
  }
}

hipError_t launch_append(const fsx_cache_desc& c, const void* k_rows, const void* v_rows, int n_rows,
                         const int64_t* first, hipStream_t s) {
  AppendArgs a{};
  const int es = c.dtype == FSX_F32 ? 4 : (c.dtype == FSX_BF16 ? 2 : 1);
  a.ks = (const uint4*)k_rows; a.vs = (const uint4*)v_rows; a.kc = (uint4*)c.k; a.vc = (uint4*)c.v;
  a.cap = c.capacity; a.row_chunks = (int64_t)c.head_dim * es / 16;
  a.n_layers = c.n_layers; a.n_heads = c.n_heads; a.n_rows = n_rows; a.B = c.batch;
  a.token_major = (c.layout & FSX_CACHE_TOKEN_MAJOR) != 0;
  for (int b = 0; b < c.batch; ++b) a.first[b] = first[b];
  const int64_t total = (int64_t)a.B * a.n_layers * a.n_heads * a.n_rows * a.row_chunks;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(k_append, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace fsx

namespace fsx {

// =====================================================================================================
// Zero fill of a device range (a kernel, not a memset, so that it is an ordinary kernel node when the caller
// captures the stream into a graph).  Whole 16-byte chunks; `bytes` is a multiple of 256.
// =====================================================================================================
__global__ __launch_bounds__(256) void k_fill_zero(uint4* p, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0, 0, 0, 0);
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  const int64_t n16 = (int64_t)(bytes / 16);
  if (n16 == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n16 + 255) / 256, 2048);
  hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(256), 0, s, (uint4*)p, n16);
  return hipGetLastError();
}

}  // namespace fsx
