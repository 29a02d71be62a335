// The whole expert tick (Sec. 3.1, Eq. (1)) as ONE persistent cooperative launch.
//
// Every workgroup (one per CU) walks the same phase sequence; within a layer
//   Q  : RMSNorm + q/k/v projection (+ rotary, q pre-scale) per 16-column tile
//   A  : joint attention per (agent, range of cached rows, head): the 4 waves split the 32-row tiles (or
//        the query tiles when there are many queries) and merge in LDS; the expert's own rows are tiles
//        of the agent's last range; when an agent's rows were split over several ranges, the last range
//        to finish merges them (log-sum-exp)
//   O  : output projection, split-K by head group; the last split of each column tile adds the
//        residual and writes h_mid plus per-tile sums of squares for the next RMSNorm
//   F1 : RMSNorm + gate/up projection with SwiGLU
//   D  : down projection, split-K; the last split adds the residual and writes h_out
// and the head pools the first T tokens at the end.  Phases are connected by per-producer flags, not
// grid barriers: a producer writes its outputs with device-coherent stores, waits for them to
// complete, and stores a flag holding a stamp that grows with (launch, layer); a consumer polls only
// the flags of the tiles it reads.  Everything produced inside the launch is read with device-coherent
// loads: a cache line written in parts by workgroups on different XCDs may sit in an L2 with some parts
// missing, and an ordinary load could hit it.  Weights and cache rows are read-only and use ordinary
// loads, and a workgroup issues its weight loads for a phase before it waits for that phase's inputs.
// Every wait is bounded in real time; on timeout the launch records a failure and the head writes NaN
// waypoints.

#include "attn_device.h"
#include "common.h"
#include "kernels.h"

namespace fsx {

constexpr int XSTR = 520;  // LDS row stride (bf16 elements) of staged activations: 512 + 8 padding
constexpr int NTHR = 256;
constexpr int UMAX = 4;    // projection units whose weights a wave holds in registers at once
constexpr int STW = 16 * 128 + 32;  // LDS floats of one wave's attention state: O[16][128], (m, l)[16]

template <int MT>
struct TickLds {
  uint16_t x[MT * 16][XSTR];  // staged activation rows (bf16) of the current M-chunk
  f32x4 red[4][MT][WAVE];     // cross-wave reduction of projection accumulators
  float st[4][STW];           // per-wave attention states
  float r[MT * 16];           // RMSNorm row scales of the chunk
  float tmp[512];             // embed / head scratch
  float red2[16][16];         // head: per-wave partial sums
  float hr[64];               // head: row scales of the pooled tokens (at most 64)
  int ok;
  int last;
};

__device__ __forceinline__ uint64_t stamp_of(const TickArgs& a, int layer, int n_layers) {
  return a.epoch * (uint64_t)(n_layers + 2) + (uint64_t)(layer + 2);
}
__device__ __forceinline__ uint64_t fail_tag(const TickArgs& a) { return a.epoch + 1; }

// Wave-level wait until flags[(i / inner) * stride + i % inner] >= target for i < n.  False on timeout or
// when another workgroup has already recorded a failure for this launch.
__device__ __forceinline__ bool wave_wait(const uint64_t* flags, int n, uint64_t target, const TickArgs& a,
                                          int inner = 1 << 30, int stride = 0) {
  const int lane = threadIdx.x & 63;
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  for (int base = 0; base < n; base += WAVE) {
    const int i = base + lane;
    const int64_t fi = (int64_t)(i / inner) * stride + i % inner;
    for (uint32_t spin = 0;; ++spin) {
      const bool ok = i >= n || ld_dev(flags + fi) >= target;
      if (__all(ok)) break;
      // back off after the first polls: many workgroups poll the same flag lines
      if (spin < 8)
        __builtin_amdgcn_s_sleep(1);
      else
        __builtin_amdgcn_s_sleep(6);
      if ((spin & 31) == 31) {
        if (__builtin_amdgcn_s_memrealtime() - t0 > a.timeout_ticks || ld_dev(a.status) == fail_tag(a)) {
          if (lane == 0) st_dev(a.status, fail_tag(a));
          return false;
        }
      }
    }
  }
  return true;
}

template <int MT>
__device__ __forceinline__ bool wg_wait(const uint64_t* flags, int n, uint64_t target, const TickArgs& a, TickLds<MT>& L,
                                        int inner = 1 << 30, int stride = 0) {
  if (threadIdx.x < WAVE) {
    const bool ok = wave_wait(flags, n, target, a, inner, stride);
    if (threadIdx.x == 0) L.ok = ok;
  }
  __syncthreads();
  const bool ok = L.ok;
  __syncthreads();
  return ok;
}

__device__ __forceinline__ void trace_mark(const TickArgs& a, int ev, int n_layers) {
  if (a.trace && threadIdx.x == 0)
    a.trace[(int64_t)blockIdx.x * trace_events(n_layers) + ev] = __builtin_amdgcn_s_memrealtime();
}

// sub-phase mark k (0..10) of layer l
#define TICK_SUB(l, k) trace_mark(a, 2 + 16 * (l) + 5 + (k), dm.n_layers)

// ------------------------------------------------------------------------------------------ staging
// Row scales of an RMSNorm input chunk: r[row] = 1/sqrt(mean(h^2) + eps) from the per-16-column sums of
// squares ssq[tile][m] (rows past `rows` get 0).  16 threads per row, a fixed-order 16-lane sum.  (The
// norm's gain is folded into the packed weights; projections scale output row m by r[m].)  With one
// wave per SIMD nothing hides a load's latency, so every step issues all of its loads before using any.
template <int MT>
__device__ __forceinline__ void load_row_scales(const float* ssq, int m0, int rows, int M, int K, float eps,
                                                TickLds<MT>& L) {
  const int tid = threadIdx.x, ntile = K / 16;  // <= 32
  const int g = tid & 15, rw = tid >> 4;
  float part[MT];
#pragma unroll
  for (int p = 0; p < MT; ++p) {
    const int i = rw + 16 * p;
    float s0 = 0.f, s1 = 0.f;
    if (i < rows) {
      if (g < ntile) s0 = ld_dev_f(ssq + (int64_t)g * M + m0 + i);
      if (g + 16 < ntile) s1 = ld_dev_f(ssq + (int64_t)(g + 16) * M + m0 + i);
    }
    part[p] = s0 + s1;
  }
#pragma unroll
  for (int p = 0; p < MT; ++p) {
    float v = part[p];
    v += shfl_xor(v, 8);
    v += shfl_xor(v, 4);
    v += shfl_xor(v, 2);
    v += shfl_xor(v, 1);
    const int i = rw + 16 * p;
    if (g == 0) L.r[i] = i < rows ? 1.0f / sqrtf(v / (float)K + eps) : 0.f;
  }
}

// x[row][k] = src[(m0+row)*ld + k] (bf16) for k < K (K/8 a power of two: shift indexing), rows past
// `rows` zero; ends with a barrier.  The source was produced inside this launch, in cache lines that
// several workgroups (on several XCDs) each wrote in part, so it is read with device-coherent loads.
template <int MT>
__device__ __forceinline__ void stage_copy(const uint16_t* src, int ld, int m0, int rows, int K, TickLds<MT>& L) {
  const int cpr = K / 8, lg = __ffs(cpr) - 1, total = MT * 16 * cpr;
  constexpr int BATCH = 8;
  for (int i0 = threadIdx.x; i0 < total; i0 += BATCH * NTHR) {
    uint4 v[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int i = i0 + k * NTHR;
      const int row = i >> lg, ch = i & (cpr - 1);
      v[k] = make_uint4(0, 0, 0, 0);
      if (i < total && row < rows) v[k] = ld_dev16(src + (int64_t)(m0 + row) * ld + ch * 8);
    }
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int i = i0 + k * NTHR;
      if (i < total) *reinterpret_cast<uint4*>(&L.x[i >> lg][(i & (cpr - 1)) * 8]) = v[k];
    }
  }
  __syncthreads();
}

// ------------------------------------------------------------------------------------------ projections
// A projection unit is one 16-column tile over a range of nkb k-blocks; wave w owns the unit's k-blocks
// i = w, w+4, w+8, w+12 (a range is at most 512 columns = 16 blocks), whose 1 KiB weight blocks it holds
// in registers.
__device__ __forceinline__ void load_unit_w(const uint4* __restrict__ wtile, int kb0, int nkb, uint4 w[4]) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = wave + 4 * j;
    w[j] = i < nkb ? wtile[(int64_t)(kb0 + i) * WAVE + lane] : make_uint4(0, 0, 0, 0);
  }
}

// acc = staged x (k-blocks 0..nkb-1 of the unit's range) times the unit's weights, summed over the 4
// waves through LDS and handed to epi(mt, C-layout values, c, grp) by wave mt % 4.
template <int MT, typename Epi>
__device__ __forceinline__ void unit_gemm(const uint4 w[4], int nkb, TickLds<MT>& L, Epi epi) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = lane & 15, grp = lane >> 4;
  f32x4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = wave + 4 * j;
    if (i < nkb) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const uint4 xa = *reinterpret_cast<const uint4*>(&L.x[mt * 16 + c][i * 32 + 8 * grp]);
        acc[mt] = mfma_bf16(xa, w[j], acc[mt]);
      }
    }
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) L.red[wave][mt][lane] = acc[mt];
  __syncthreads();
  for (int mt = wave; mt < MT; mt += 4) {
    const f32x4 s = L.red[0][mt][lane] + L.red[1][mt][lane] + L.red[2][mt][lane] + L.red[3][mt][lane];
    epi(mt, s, c, grp);
  }
  __syncthreads();
}

// Last split of a column tile: h_dst[m][tile] = h_src[m][tile] + sum_s part[s][m][tile] (fixed order), also
// as bf16 in hb_dst, and ssq_dst[tile][m] = sum over the tile of h_dst^2; resets the tile's counter and
// publishes its flag.
__device__ __forceinline__ void reduce_tile(const TickArgs& a, const TickParams& tp, const Dims& dm, int nt, int nsplit,
                                            const float* h_src, float* h_dst, uint16_t* hb_dst, float* ssq_dst,
                                            uint32_t* cnt, uint64_t* flag, uint64_t st) {
  const int M = tp.M, d = dm.d, total = M * 16;
  constexpr int BATCH = 2;
  for (int i0 = threadIdx.x; i0 < total; i0 += BATCH * NTHR) {
    float p[BATCH][8], hv[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int idx = i0 + k * NTHR;
      const int m = idx >> 4, n = nt * 16 + (idx & 15);
      const bool in = idx < total;
      hv[k] = in ? ld_dev_f(h_src + (int64_t)m * d + n) : 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s) p[k][s] = in && s < nsplit ? ld_dev_f(a.part + ((int64_t)s * M + m) * d + n) : 0.f;
    }
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int idx = i0 + k * NTHR;
      const int m = idx >> 4, c = idx & 15, n = nt * 16 + c;
      float acc = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s) acc += p[k][s];
      const float v = hv[k] + acc;
      if (idx < total) st_dev_f(h_dst + (int64_t)m * d + n, v);
      const float vn = shfl_xor(v, 1);
      if (idx < total && (c & 1) == 0) st_dev(reinterpret_cast<uint32_t*>(hb_dst + (int64_t)m * d + n), pack_bf16x2(v, vn));
      float sq = v * v;
      sq += shfl_xor(sq, 8);
      sq += shfl_xor(sq, 4);
      sq += shfl_xor(sq, 2);
      sq += shfl_xor(sq, 1);
      if (c == 0 && idx < total) st_dev_f(ssq_dst + (int64_t)nt * M + m, sq);
    }
  }
  if (threadIdx.x == 0) st_dev(cnt + nt, 0u);
  stores_done();
  __syncthreads();
  if (threadIdx.x == 0) st_dev(flag + nt, st);
}

// ------------------------------------------------------------------------------------------ embed
template <int MT>
__device__ __forceinline__ void phase_embed(const TickArgs& a, const TickParams& tp, const Dims& dm, TickLds<MT>& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, half = dm.Dh / 2;
  const uint64_t st = stamp_of(a, -1, dm.n_layers);
  for (int m = blockIdx.x; m < M; m += G) {
    const int b = m / tp.S, t = m % tp.S;
    for (int n = 2 * threadIdx.x; n < d; n += 2 * NTHR) {  // two channels per thread (d is even)
      const int64_t idx = (int64_t)m * d + n;
      float v0, v1;
      if (a.tok_dtype == FSX_BF16) {
        const uint32_t pr = *reinterpret_cast<const uint32_t*>((const uint16_t*)a.tokens + idx);
        v0 = bf16_to_f32((uint16_t)(pr & 0xffffu));
        v1 = bf16_to_f32((uint16_t)(pr >> 16));
      } else {
        v0 = ((const float*)a.tokens)[idx];
        v1 = ((const float*)a.tokens)[idx + 1];
      }
      st_dev(reinterpret_cast<uint64_t*>(a.h0 + idx), (uint64_t)__float_as_uint(v0) | ((uint64_t)__float_as_uint(v1) << 32));
      st_dev(reinterpret_cast<uint32_t*>(a.hb0 + idx), pack_bf16x2(v0, v1));
      L.tmp[n] = v0 * v0;
      L.tmp[n + 1] = v1 * v1;
    }
    for (int j = threadIdx.x; j < half; j += NTHR) {
      double cs = 1.0, sn = 0.0;
      if (dm.rope_base > 0.f) {
        const double ang = (double)(tp.pos[b] + t) * pow((double)dm.rope_base, -2.0 * (double)j / (double)dm.Dh);
        cs = cos(ang);
        sn = sin(ang);
      }
      st_dev_f(a.rope + ((int64_t)m * half + j) * 2, (float)cs);
      st_dev_f(a.rope + ((int64_t)m * half + j) * 2 + 1, (float)sn);
    }
    // return the last-arriver counters to zero (robust to an earlier launch that stopped midway)
    for (int i = m * NTHR + threadIdx.x; i < a.n_att_cnt; i += M * NTHR) st_dev(a.att_cnt + i, 0u);
    if (m == 0)
      for (int i = threadIdx.x; i < d / 16; i += NTHR) {
        st_dev(a.o_cnt + i, 0u);
        st_dev(a.d_cnt + i, 0u);
      }
    __syncthreads();
    for (int tile = threadIdx.x; tile < d / 16; tile += NTHR) {
      float s = 0.f;
      for (int c = 0; c < 16; ++c) s += L.tmp[tile * 16 + c];
      st_dev_f(a.ssq0 + (int64_t)tile * M + m, s);
    }
    stores_done();
    __syncthreads();
    if (threadIdx.x == 0) st_dev(a.f_embed + m, st);
  }
}

// ------------------------------------------------------------------------------------------ Q
template <int MT>
__device__ __forceinline__ bool phase_qkv(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds<MT>& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, A = dm.A, Dh = dm.Dh, half = Dh / 2;
  const int n_units = 3 * A / 16;
  const TickLayer& W = a.layers[l];
  const int KB = d / 32;
  const float qs = LOG2E / sqrtf((float)Dh);
  const uint16_t* hbsrc = l == 0 ? a.hb0 : a.hbout + (int64_t)(l - 1) * M * d;
  const float* ssq = l == 0 ? a.ssq0 : a.ssq_out + (int64_t)(l - 1) * (d / 16) * M;
  bool waited = false;
  for (int u0 = blockIdx.x; u0 < n_units; u0 += UMAX * G) {
    uint4 w[UMAX][4];
#pragma unroll
    for (int k = 0; k < UMAX; ++k) {
      const int u = u0 + k * G;
      if (u < n_units) load_unit_w(W.wqkv + (int64_t)u * KB * WAVE, 0, KB, w[k]);
    }
    if (!waited) {
      TICK_SUB(l, 0);
      const bool ok = l == 0 ? wg_wait(a.f_embed, M, stamp_of(a, -1, dm.n_layers), a, L)
                             : wg_wait(a.f_hout, d / 16, stamp_of(a, l - 1, dm.n_layers), a, L);
      if (!ok) return false;
      waited = true;
      TICK_SUB(l, 1);
    }
    for (int m0 = 0; m0 < M; m0 += MT * 16) {
      const int rows = min(MT * 16, M - m0);
      load_row_scales<MT>(ssq, m0, rows, M, d, dm.eps, L);
      stage_copy<MT>(hbsrc, d, m0, rows, d, L);
      TICK_SUB(l, 2);
#pragma unroll
      for (int k = 0; k < UMAX; ++k) {
        const int u = u0 + k * G;
        if (u >= n_units) break;
        const int sec = (u * 16) / A;  // 0 q, 1 k, 2 v
        const int nl0 = u * 16 - sec * A;
        unit_gemm<MT>(w[k], KB, L, [&](int mt, f32x4 s, int c, int grp) {
          const int nl = nl0 + c;
          if (sec == 2) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int row = m0 + mt * 16 + 4 * grp + i;
              s[i] *= L.r[mt * 16 + 4 * grp + i];  // RMSNorm row scale
              const float other = shfl_xor(s[i], 1);
              if ((c & 1) == 0 && row < M)
                st_dev(reinterpret_cast<uint32_t*>(a.vself + (int64_t)row * A + nl), pack_bf16x2(s[i], other));
            }
          } else {
            const int head = nl / Dh, p = nl % Dh;
            const int j = 8 * (p / 16) + (c & 7);
            const int dch = c < 8 ? j : half + j;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              s[i] *= L.r[mt * 16 + 4 * grp + i];  // RMSNorm row scale
              const float partner = shfl_xor(s[i], 8);
              const int row = m0 + mt * 16 + 4 * grp + i;
              const int rrow = row < M ? row : 0;
              // rope rows (Dh*4 bytes, line aligned) have one producer each and are complete before any
              // projection starts, so ordinary loads cannot see a partial line
              const float cs = a.rope[((int64_t)rrow * half + j) * 2 + 0];
              const float sn = a.rope[((int64_t)rrow * half + j) * 2 + 1];
              const float r = c < 8 ? s[i] * cs - partner * sn : s[i] * cs + partner * sn;
              const int64_t o = (int64_t)row * A + head * Dh + dch;
              if (sec == 0) {
                if (row < M) st_dev_f(a.q + o, r * qs);
              } else {
                const float nb = shfl_xor(r, 1);  // neighbouring channel dch+1 sits in lane c+1
                if ((c & 1) == 0 && row < M) st_dev(reinterpret_cast<uint32_t*>(a.kself + o), pack_bf16x2(r, nb));
              }
            }
          }
        });
      }
    }
  }
  TICK_SUB(l, 3);
  stores_done();
  __syncthreads();
  TICK_SUB(l, 4);
  if (threadIdx.x == 0) {
    const uint64_t st = stamp_of(a, l, dm.n_layers);
    for (int u = blockIdx.x; u < n_units; u += G) st_dev(a.f_qkv + u, st);
  }
  return true;
}

// ------------------------------------------------------------------------------------------ A
// One 32-row tile of one row source, as MFMA operands: kf[rt*4 + kb] = K rows r0+16rt+c, channels
// 32kb+8grp..; vr[j] = V row r0 + (j<4 ? 4grp+j : 16+4grp+j-4), channels 8c..8c+7.  Rows past i1 load row
// i0 (they are masked out of the softmax).
template <int KT, bool RING, bool COH>
__device__ __forceinline__ void tile_load(const char* kb, const char* vb, int64_t row_bytes, int64_t start,
                                          int64_t cap, int i0, int r0, int i1, uint4 kf[8], uint4 vr[8]) {
  constexpr int ES = KT == 0 ? 2 : 1;
  const int lane = threadIdx.x & 63, c = lane & 15, grp = lane >> 4;
  auto roff = [&](int i) -> int64_t {
    int64_t slot = i;
    if (RING) {
      slot = start + i;
      if (slot >= cap) slot -= cap;
    }
    return slot * row_bytes;
  };
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int i = r0 + 16 * rt + c;
    const char* p = kb + roff(i < i1 ? i : i0);
#pragma unroll
    for (int k = 0; k < 4; ++k) kf[rt * 4 + k] = load8<KT, COH>(p + (32 * k + 8 * grp) * ES);
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int rr = r0 + (j < 4 ? 4 * grp + j : 16 + 4 * grp + (j - 4));
    vr[j] = load8<KT, COH>(vb + roff(rr < i1 ? rr : i0) + 8 * c * ES);
  }
}

// online-softmax update of (o, m_run, l_run) with one tile; F16 selects fp16 operands, kscale multiplies
// the scores and vscale the probabilities that weight V (fp8 rows carry their scales here).
template <bool F16>
__device__ __forceinline__ void tile_compute(const uint4 kf[8], const uint4 vr[8], const uint4 qf[4], int r0,
                                             int i1, float kscale, float vscale, f32x4 o[8], float& m_run,
                                             float& l_run) {
  const int lane = threadIdx.x & 63, grp = lane >> 4;
  f32x4 s[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    s[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < 4; ++k) s[rt] = F16 ? mfma_f16(kf[rt * 4 + k], qf[k], s[rt]) : mfma_bf16(kf[rt * 4 + k], qf[k], s[rt]);
  }
  float mx = -INFINITY;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = r0 + 16 * rt + 4 * grp + i;
      const float v = rr < i1 ? s[rt][i] * kscale : -INFINITY;
      s[rt][i] = v;
      mx = fmaxf(mx, v);
    }
  mx = fmaxf(mx, shfl_xor(mx, 16));
  mx = fmaxf(mx, shfl_xor(mx, 32));
  const float m_new = fmaxf(m_run, mx);
  const float alpha = exp2f(m_run - m_new);
  float p[8], ps = 0.f;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[rt * 4 + i] = exp2f(s[rt][i] - m_new);
      ps += p[rt * 4 + i];
    }
  l_run = l_run * alpha + ps;
  m_run = m_new;
  uint4 pf;
  if (F16)
    pf = make_uint4(pack_f16x2(p[0] * vscale, p[1] * vscale), pack_f16x2(p[2] * vscale, p[3] * vscale),
                    pack_f16x2(p[4] * vscale, p[5] * vscale), pack_f16x2(p[6] * vscale, p[7] * vscale));
  else
    pf = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7]));
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a_i = shfl(alpha, 4 * grp + i);
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k][i] *= a_i;
  }
  uint4 vt[8];
  transpose8x8_b16(vr, vt);
#pragma unroll
  for (int k = 0; k < 8; ++k) o[k] = F16 ? mfma_f16(pf, vt[k], o[k]) : mfma_bf16(pf, vt[k], o[k]);
}

// Describes the tiles of one attention unit: cache rows [i0, i1) then (last range only) the S own rows.
struct AUnit {
  int b, h, r, nr;
  int i0, i1;       // cache rows of this range
  int nct, nst;     // cache tiles, own-row tiles
  const char* kc;   // cache K/V base of (b, layer, head) (slot 0)
  const char* vc;
  const char* ks;   // own rows base of (b, head)
  const char* vs;
  float ksc, vsc;   // fp8 scales
};

// Process tiles j = part, part+step, ... of the unit for query tile tt; returns the wave's state.
template <int KT>
__device__ __forceinline__ void attn_tiles(const TickArgs& a, const TickParams& tp, const Dims& dm, const AUnit& U, int tt,
                           int part, int step, uint64_t st, bool& ok, f32x4 o[8], float& m_run, float& l_run) {
  constexpr int ES = KT == 0 ? 2 : 1;
  const int lane = threadIdx.x & 63, grp = lane >> 4;
  const int A = dm.A, Dh = dm.Dh;
  const int ntiles = U.nct + U.nst;
#pragma unroll
  for (int k = 0; k < 8; ++k) o[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  m_run = -INFINITY;
  l_run = 0.f;
  if (part >= ntiles) return;
  const int64_t crow = (int64_t)Dh * ES, srow = (int64_t)A * 2;
  uint4 kf[8], vr[8];
  // the first tile, when it is a cache tile, does not depend on this layer's projections: load it now
  int j = part;
  if (j < U.nct) tile_load<KT, true, false>(U.kc, U.vc, crow, tp.start[U.b], a.cv.cap, U.i0, U.i0 + 32 * j, U.i1, kf, vr);
  const int qt = U.h * (Dh / 16);
  ok = wave_wait(a.f_qkv + qt, Dh / 16, st, a);
  bool mine_self = false;
  for (int jj = part; jj < ntiles; jj += step) mine_self = mine_self || jj >= U.nct;
  if (ok && mine_self)
    ok = wave_wait(a.f_qkv + A / 16 + qt, Dh / 16, st, a) && wave_wait(a.f_qkv + 2 * A / 16 + qt, Dh / 16, st, a);
  if (!ok) return;
  const int t = tt * 16 + (lane & 15);
  const bool tv = t < tp.S;
  const int64_t qrow = ((int64_t)U.b * tp.S + (tv ? t : 0)) * A + (int64_t)U.h * Dh;
  uint4 qb[4], qh[4];
  load_q_frag<0, true>(a.q, qrow, tv, grp, qb);
  if (KT == 1) load_q_frag<1, true>(a.q, qrow, tv, grp, qh);
  if (j >= U.nct) tile_load<0, false, true>(U.ks, U.vs, srow, 0, 0, 0, 32 * (j - U.nct), tp.S, kf, vr);
  for (; j < ntiles; j += step) {
    const int jn = j + step;
    uint4 kn[8], vn[8];
    if (jn < U.nct)
      tile_load<KT, true, false>(U.kc, U.vc, crow, tp.start[U.b], a.cv.cap, U.i0, U.i0 + 32 * jn, U.i1, kn, vn);
    else if (jn < ntiles)
      tile_load<0, false, true>(U.ks, U.vs, srow, 0, 0, 0, 32 * (jn - U.nct), tp.S, kn, vn);
    if (j < U.nct) {
      if (KT == 1)
        tile_compute<true>(kf, vr, qh, U.i0 + 32 * j, U.i1, U.ksc, U.vsc, o, m_run, l_run);
      else
        tile_compute<false>(kf, vr, qb, U.i0 + 32 * j, U.i1, 1.f, 1.f, o, m_run, l_run);
    } else {
      tile_compute<false>(kf, vr, qb, 32 * (j - U.nct), tp.S, 1.f, 1.f, o, m_run, l_run);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      kf[k] = kn[k];
      vr[k] = vn[k];
    }
  }
}

// write a wave's state (o in the PV C layout, m and the lane-partial l) to LDS slot w
__device__ __forceinline__ void state_to_lds(float* stw, const f32x4 o[8], float m_run, float l_run) {
  const int lane = threadIdx.x & 63, c = lane & 15, grp = lane >> 4;
  float lt = l_run + shfl_xor(l_run, 16);
  lt += shfl_xor(lt, 32);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int k = 0; k < 8; ++k) stw[(4 * grp + i) * 128 + 8 * c + k] = o[k][i];
  if (grp == 0) {
    stw[2048 + 2 * c] = m_run;
    stw[2048 + 2 * c + 1] = lt;
  }
}

// Merge LDS states of waves [w0, w0+nw) for query tile tt: each thread owns (t, 8 channels).  If final,
// normalise into the attention output; else store the unnormalised partial of slot `item`.
template <int MT>
__device__ __forceinline__ void merge_states(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, const AUnit& U, int tt,
                             int w0, int nw, bool final_out, int64_t item, TickLds<MT>& L) {
  const int t = threadIdx.x >> 4, d0 = (threadIdx.x & 15) * 8;
  float Mx = -INFINITY;
  for (int w = 0; w < nw; ++w) Mx = fmaxf(Mx, L.st[w0 + w][2048 + 2 * t]);
  float Ls = 0.f, acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.f;
  for (int w = 0; w < nw; ++w) {
    const float* stw = L.st[w0 + w];
    const float f = Mx == -INFINITY ? 0.f : exp2f(stw[2048 + 2 * t] - Mx);
    Ls += stw[2048 + 2 * t + 1] * f;
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += stw[t * 128 + d0 + k] * f;
  }
  if (final_out) {
    const int tok = tt * 16 + t;
    if (tok < tp.S) {
      const float inv = 1.0f / Ls;
      uint16_t* dst = a.attn + (int64_t)l * tp.M * dm.A + ((int64_t)U.b * tp.S + tok) * dm.A + (int64_t)U.h * dm.Dh + d0;
      st_dev16(dst, make_uint4(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                               pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)));
    }
  } else {
    float* po = a.att_o + (item * 16 + t) * 128 + d0;
    st_dev_f4(po, make_float4(acc[0], acc[1], acc[2], acc[3]));
    st_dev_f4(po + 4, make_float4(acc[4], acc[5], acc[6], acc[7]));
    if ((threadIdx.x & 15) == 0) {
      st_dev_f(a.att_ml + item * 32 + 2 * t, Mx);
      st_dev_f(a.att_ml + item * 32 + 2 * t + 1, Ls);
    }
  }
}

// the last range of an agent to finish merges the partials of all its ranges (fixed order)
template <int MT>
__device__ __forceinline__ void combine_ranges(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, const AUnit& U) {
  const int t = threadIdx.x >> 4, d0 = (threadIdx.x & 15) * 8;
  const int H = dm.H;
  for (int tt = 0; tt < tp.n_tt; ++tt) {
    float Mx = -INFINITY, Ls = 0.f, acc[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = 0.f;
#pragma unroll 2
    for (int r = 0; r < U.nr; ++r) {
      const int64_t item = ((int64_t)(tp.range_prefix[U.b] + r) * H + U.h) * tp.n_tt + tt;  // pair * n_tt + tt
      const float ms = ld_dev_f(a.att_ml + item * 32 + 2 * t), ls = ld_dev_f(a.att_ml + item * 32 + 2 * t + 1);
      const float* po = a.att_o + (item * 16 + t) * 128 + d0;
      const float4 v0 = ld_dev_f4(po), v1 = ld_dev_f4(po + 4);
      const float mn = fmaxf(Mx, ms);
      const float fa = Mx == -INFINITY ? 0.f : exp2f(Mx - mn), fb = ms == -INFINITY ? 0.f : exp2f(ms - mn);
      Ls = Ls * fa + ls * fb;
      acc[0] = acc[0] * fa + v0.x * fb; acc[1] = acc[1] * fa + v0.y * fb;
      acc[2] = acc[2] * fa + v0.z * fb; acc[3] = acc[3] * fa + v0.w * fb;
      acc[4] = acc[4] * fa + v1.x * fb; acc[5] = acc[5] * fa + v1.y * fb;
      acc[6] = acc[6] * fa + v1.z * fb; acc[7] = acc[7] * fa + v1.w * fb;
      Mx = mn;
    }
    const int tok = tt * 16 + t;
    if (tok < tp.S) {
      const float inv = 1.0f / Ls;
      uint16_t* dst = a.attn + (int64_t)l * tp.M * dm.A + ((int64_t)U.b * tp.S + tok) * dm.A + (int64_t)U.h * dm.Dh + d0;
      st_dev16(dst, make_uint4(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                               pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)));
    }
  }
}

// Attention units are (agent, range, head, query tile).  Pairs (agent range, head) come in groups of 8 and a
// group's units are ordered query tile by query tile, so unit u runs on workgroup u mod G and the query
// tiles of one pair land on the same XCD (u = 8*n_tt*grp + 8*tt + j): they read the same cached rows
// through that XCD's L2.
template <int MT, int KT>
__device__ __forceinline__ bool phase_attn(const TickArgs& a, const TickParams& tp, const Dims& dm, int l,
                                           TickLds<MT>& L) {
  constexpr int ES = KT == 0 ? 2 : 1;
  const int G = gridDim.x, wave = threadIdx.x >> 6;
  const int H = dm.H, Dh = dm.Dh, A = dm.A, n_tt = tp.n_tt;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const int n_pairs = tp.range_prefix[tp.B] * H;
  const int n_units = n_tt == 1 ? n_pairs : (n_pairs + 7) / 8 * 8 * n_tt;
  for (int u = blockIdx.x; u < n_units; u += G) {
    int pair = u, tt = 0;
    if (n_tt > 1) {
      const int grp = u / (8 * n_tt), rem = u % (8 * n_tt);
      tt = rem / 8;
      pair = 8 * grp + rem % 8;
      if (pair >= n_pairs) continue;
    }
    AUnit U;
    U.h = pair % H;
    const int slot = pair / H;
    int b = 0;
    while (b + 1 < tp.B && tp.range_prefix[b + 1] <= slot) ++b;
    U.b = b;
    U.r = slot - tp.range_prefix[b];
    U.nr = tp.range_prefix[b + 1] - tp.range_prefix[b];
    U.i0 = U.r * tp.range_rows;
    U.i1 = min(U.i0 + tp.range_rows, tp.len[b]);
    U.nct = U.i1 > U.i0 ? (U.i1 - U.i0 + 31) / 32 : 0;
    U.nst = U.r == U.nr - 1 ? (tp.S + 31) / 32 : 0;
    const int64_t slab = (((int64_t)b * a.cv.n_layers + l) * H + U.h) * a.cv.cap;  // head-major (b, l, h) ring
    U.kc = (const char*)a.cv.k + slab * Dh * ES;
    U.vc = (const char*)a.cv.v + slab * Dh * ES;
    U.ks = (const char*)a.kself + ((int64_t)b * tp.S * A + (int64_t)U.h * Dh) * 2;
    U.vs = (const char*)a.vself + ((int64_t)b * tp.S * A + (int64_t)U.h * Dh) * 2;
    U.ksc = U.vsc = 1.f;
    if (KT == 1) {
      const int64_t si = ((int64_t)b * a.cv.n_layers + l) * H + U.h;
      U.ksc = a.cv.k_scale[si];
      U.vsc = a.cv.v_scale[si];
    }
    const bool final_out = U.nr == 1;
    bool ok = true;
    f32x4 o[8];
    float m_run, l_run;
    const bool first_unit = u == (int)blockIdx.x;
    attn_tiles<KT>(a, tp, dm, U, tt, wave, 4, st, ok, o, m_run, l_run);
    state_to_lds(L.st[wave], o, m_run, l_run);
    if (!ok && (threadIdx.x & 63) == 0) L.ok = 0;
    __syncthreads();
    if (first_unit) TICK_SUB(l, 5);
    if (!L.ok) return false;
    merge_states<MT>(a, tp, dm, l, U, tt, 0, 4, final_out, (int64_t)(pair * n_tt + tt), L);
    stores_done();
    __syncthreads();
    if (first_unit) TICK_SUB(l, 6);
    const int ci = b * H + U.h;
    // a pair is complete when its n_tt query tiles (and, with several ranges, all its ranges) are written
    const uint32_t need = (uint32_t)(U.nr * n_tt);
    if (threadIdx.x == 0) L.last = need == 1 ? 1 : atomic_add_dev(a.att_cnt + ci, 1u) == need - 1;
    __syncthreads();
    if (L.last) {
      if (!final_out) combine_ranges<MT>(a, tp, dm, l, U);
      if (threadIdx.x == 0 && need > 1) st_dev(a.att_cnt + ci, 0u);
      stores_done();
      __syncthreads();
      if (threadIdx.x == 0) st_dev(a.f_attn + ci, st);
    }
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------------------------------ O
template <int MT>
__device__ __forceinline__ bool phase_oproj(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds<MT>& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, A = dm.A, H = dm.H;
  const int ntiles = d / 16, n_units = ntiles * a.ks_o;
  const int hps = H / a.ks_o, nk = A / a.ks_o, nkb = nk / 32;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const TickLayer& W = a.layers[l];
  const uint16_t* attn = a.attn + (int64_t)l * M * A;
  const float* hin = l == 0 ? a.h0 : a.hout + (int64_t)(l - 1) * M * d;
  for (int u = blockIdx.x; u < n_units; u += G) {
    const int nt = u % ntiles, ks = u / ntiles;
    uint4 w[4];
    load_unit_w(W.wo + (int64_t)nt * (A / 32) * WAVE, ks * nkb, nkb, w);
    if (!wg_wait(a.f_attn + ks * hps, tp.B * hps, st, a, L, hps, H)) return false;
    if (u == (int)blockIdx.x) TICK_SUB(l, 7);
    for (int m0 = 0; m0 < M; m0 += MT * 16) {
      const int rows = min(MT * 16, M - m0);
      stage_copy<MT>(attn + ks * nk, A, m0, rows, nk, L);
      unit_gemm<MT>(w, nkb, L, [&](int mt, f32x4 s, int c, int grp) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = m0 + mt * 16 + 4 * grp + i;
          if (row < M) st_dev_f(a.part + ((int64_t)ks * M + row) * d + nt * 16 + c, s[i]);
        }
      });
    }
    stores_done();
    __syncthreads();
    if (u == (int)blockIdx.x) TICK_SUB(l, 8);
    if (threadIdx.x == 0) L.last = atomic_add_dev(a.o_cnt + nt, 1u) == (uint32_t)(a.ks_o - 1);
    __syncthreads();
    if (u == (int)blockIdx.x) TICK_SUB(l, 9);
    if (L.last)
      reduce_tile(a, tp, dm, nt, a.ks_o, hin, a.hmid + (int64_t)l * M * d, a.hbmid + (int64_t)l * M * d,
                  a.ssq_mid + (int64_t)l * (d / 16) * M, a.o_cnt, a.f_hmid, st);
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------------------------------ F1
template <int MT>
__device__ __forceinline__ bool phase_gateup(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds<MT>& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, F = dm.F;
  const int n_units = 2 * F / 16;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const TickLayer& W = a.layers[l];
  const uint16_t* hbmid = a.hbmid + (int64_t)l * M * d;
  const float* ssq = a.ssq_mid + (int64_t)l * (d / 16) * M;
  uint16_t* z = a.z + (int64_t)l * M * F;
  const int KB = d / 32;
  bool waited = false;
  for (int u0 = blockIdx.x; u0 < n_units; u0 += UMAX * G) {
    uint4 w[UMAX][4];
#pragma unroll
    for (int k = 0; k < UMAX; ++k) {
      const int u = u0 + k * G;
      if (u < n_units) load_unit_w(W.wgu + (int64_t)u * KB * WAVE, 0, KB, w[k]);
    }
    if (!waited) {
      if (!wg_wait(a.f_hmid, d / 16, st, a, L)) return false;
      waited = true;
    }
    for (int m0 = 0; m0 < M; m0 += MT * 16) {
      const int rows = min(MT * 16, M - m0);
      load_row_scales<MT>(ssq, m0, rows, M, d, dm.eps, L);
      stage_copy<MT>(hbmid, d, m0, rows, d, L);
#pragma unroll
      for (int k = 0; k < UMAX; ++k) {
        const int u = u0 + k * G;
        if (u >= n_units) break;
        unit_gemm<MT>(w[k], KB, L, [&](int mt, f32x4 s, int c, int grp) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            s[i] *= L.r[mt * 16 + 4 * grp + i];  // RMSNorm row scale
            const float up = shfl_xor(s[i], 8);
            const float gt = s[i];
            const float zz = gt / (1.0f + expf(-gt)) * up;
            const float zn = shfl_xor(zz, 1);
            const int row = m0 + mt * 16 + 4 * grp + i;
            if (c < 8 && (c & 1) == 0 && row < M)
              st_dev(reinterpret_cast<uint32_t*>(z + (int64_t)row * F + u * 8 + c), pack_bf16x2(zz, zn));
          }
        });
      }
    }
  }
  stores_done();
  __syncthreads();
  if (threadIdx.x == 0)
    for (int u = blockIdx.x; u < n_units; u += G) st_dev(a.f_z + u, st);
  return true;
}

// ------------------------------------------------------------------------------------------ D
template <int MT>
__device__ __forceinline__ bool phase_down(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds<MT>& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, F = dm.F;
  const int ntiles = d / 16, n_units = ntiles * a.ks_d, nk = F / a.ks_d, nkb = nk / 32;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const TickLayer& W = a.layers[l];
  const uint16_t* z = a.z + (int64_t)l * M * F;
  const float* hmid = a.hmid + (int64_t)l * M * d;
  for (int u = blockIdx.x; u < n_units; u += G) {
    const int nt = u % ntiles, ks = u / ntiles;
    uint4 w[4];
    load_unit_w(W.wd + (int64_t)nt * (F / 32) * WAVE, ks * nkb, nkb, w);
    if (!wg_wait(a.f_z + ks * nk / 8, nk / 8, st, a, L)) return false;
    for (int m0 = 0; m0 < M; m0 += MT * 16) {
      const int rows = min(MT * 16, M - m0);
      stage_copy<MT>(z + ks * nk, F, m0, rows, nk, L);
      unit_gemm<MT>(w, nkb, L, [&](int mt, f32x4 s, int c, int grp) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = m0 + mt * 16 + 4 * grp + i;
          if (row < M) st_dev_f(a.part + ((int64_t)ks * M + row) * d + nt * 16 + c, s[i]);
        }
      });
    }
    stores_done();
    __syncthreads();
    if (threadIdx.x == 0) L.last = atomic_add_dev(a.d_cnt + nt, 1u) == (uint32_t)(a.ks_d - 1);
    __syncthreads();
    if (L.last)
      reduce_tile(a, tp, dm, nt, a.ks_d, hmid, a.hout + (int64_t)l * M * d, a.hbout + (int64_t)l * M * d,
                  a.ssq_out + (int64_t)l * (d / 16) * M, a.d_cnt, a.f_hout, st);
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------------------------------ head
// wp[b] = mean over t < T of RMSNorm(h[b][t]) * g_final, times W_head^T.  Thread tid owns columns tid and
// tid + 256 and holds the pooled rows in registers (16 rows per pass).
template <int MT>
__device__ __forceinline__ void phase_head(const TickArgs& a, const TickParams& tp, const Dims& dm, bool ok,
                                           TickLds<MT>& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, nl = dm.n_layers, T = tp.T;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  for (int b = blockIdx.x; b < tp.B; b += G) {
    if (ok) ok = wg_wait(a.f_hout, d / 16, stamp_of(a, nl - 1, nl), a, L);
    if (!ok) {
      for (int o = tid; o < dm.n_out; o += NTHR) a.waypoints[(int64_t)b * dm.n_out + o] = __builtin_nanf("");
      continue;
    }
    const float* h = a.hout + (int64_t)(nl - 1) * M * d + (int64_t)b * tp.S * d;
    const int n0 = tid, n1 = tid + NTHR;
    float xm0 = 0.f, xm1 = 0.f;
    for (int t0 = 0; t0 < T; t0 += 16) {
      float v0[16], v1[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const bool in = t0 + t < T;
        v0[t] = in && n0 < d ? ld_dev_f(h + (int64_t)(t0 + t) * d + n0) : 0.f;
        v1[t] = in && n1 < d ? ld_dev_f(h + (int64_t)(t0 + t) * d + n1) : 0.f;
      }
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        float s = v0[t] * v0[t] + v1[t] * v1[t];
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) s += shfl_xor(s, m);
        if (lane == 0) L.red2[wave][t] = s;
      }
      __syncthreads();
      if (tid < 16) {
        float s = 0.f;
        for (int w = 0; w < NTHR / WAVE; ++w) s += L.red2[w][tid];
        L.hr[tid] = 1.0f / sqrtf(s / (float)d + dm.eps);
      }
      __syncthreads();
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        if (t0 + t < T) {
          xm0 += v0[t] * L.hr[t];
          xm1 += v1[t] * L.hr[t];
        }
      }
      __syncthreads();
    }
    float* xm = L.tmp;
    if (n0 < d) xm[n0] = xm0 * a.final_norm[n0] / (float)T;
    if (n1 < d) xm[n1] = xm1 * a.final_norm[n1] / (float)T;
    __syncthreads();
    for (int o = wave; o < dm.n_out; o += NTHR / WAVE) {
      float acc = 0.f;
      for (int n = lane; n < d; n += WAVE) {
        const float wv = a.head_dtype == FSX_BF16 ? bf16_to_f32(((const uint16_t*)a.head_w)[(int64_t)o * d + n])
                                                 : ((const float*)a.head_w)[(int64_t)o * d + n];
        acc += xm[n] * wv;
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) acc += shfl_xor(acc, m);
      if (lane == 0) a.waypoints[(int64_t)b * dm.n_out + o] = acc;
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------------------------------ kernel
template <int MT, int KT>
__global__ __launch_bounds__(NTHR, 1) void k_tick(TickArgs a, TickParams tp, Dims dm) {
  __shared__ TickLds<MT> L;
  const int nl = dm.n_layers;
  trace_mark(a, 0, nl);
  if (threadIdx.x == 0) L.ok = 1;
  __syncthreads();
  phase_embed<MT>(a, tp, dm, L);
  trace_mark(a, 1, nl);
  bool ok = true;
  for (int l = 0; l < nl && ok; ++l) {
    ok = phase_qkv<MT>(a, tp, dm, l, L);
    trace_mark(a, 2 + 16 * l, nl);
    ok = ok && phase_attn<MT, KT>(a, tp, dm, l, L);
    trace_mark(a, 3 + 16 * l, nl);
    ok = ok && phase_oproj<MT>(a, tp, dm, l, L);
    trace_mark(a, 4 + 16 * l, nl);
    ok = ok && phase_gateup<MT>(a, tp, dm, l, L);
    trace_mark(a, 5 + 16 * l, nl);
    ok = ok && phase_down<MT>(a, tp, dm, l, L);
    trace_mark(a, 6 + 16 * l, nl);
  }
  phase_head<MT>(a, tp, dm, ok, L);
  trace_mark(a, 2 + 16 * nl, nl);
}

template <int KT>
static hipError_t launch_tick_kt(const TickArgs& a, const TickParams& tp, const Dims& dm, int mt, int grid,
                                 hipStream_t s) {
  void* args[] = {(void*)&a, (void*)&tp, (void*)&dm};
  const void* f = nullptr;
  switch (mt) {
    case 1: f = (const void*)k_tick<1, KT>; break;
    case 2: f = (const void*)k_tick<2, KT>; break;
    case 3: f = (const void*)k_tick<3, KT>; break;
    case 4: f = (const void*)k_tick<4, KT>; break;
    default: f = (const void*)k_tick<5, KT>; break;
  }
  return hipLaunchCooperativeKernel(f, dim3(grid), dim3(NTHR), args, 0, s);
}

int tick_mt(int M) {
  const int n_mt = (M + 15) / 16;
  const int chunks = (n_mt + 4) / 5;
  return (n_mt + chunks - 1) / chunks;
}

hipError_t tick_occupancy(int mt, int kt, int* blocks_per_cu) {
  const void* f = nullptr;
  if (kt == 0) {
    const void* fs[5] = {(const void*)k_tick<1, 0>, (const void*)k_tick<2, 0>, (const void*)k_tick<3, 0>,
                         (const void*)k_tick<4, 0>, (const void*)k_tick<5, 0>};
    f = fs[mt - 1];
  } else {
    const void* fs[5] = {(const void*)k_tick<1, 1>, (const void*)k_tick<2, 1>, (const void*)k_tick<3, 1>,
                         (const void*)k_tick<4, 1>, (const void*)k_tick<5, 1>};
    f = fs[mt - 1];
  }
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, f, NTHR, 0);
}

hipError_t launch_tick(const TickArgs& a, const TickParams& tp, const Dims& dm, int grid, hipStream_t s) {
  const int mt = tick_mt(tp.M);
  return a.cv.dtype == FSX_FP8_E4M3 ? launch_tick_kt<1>(a, tp, dm, mt, grid, s)
                                    : launch_tick_kt<0>(a, tp, dm, mt, grid, s);
}

}  // namespace fsx
