// The whole expert tick (Sec. 3.1, Eq. (1)) as ONE persistent cooperative launch.
//
// Every workgroup (one per CU) walks the same phase sequence; within a layer
//   Q  : RMSNorm + q/k/v projection (+ rotary, q pre-scale) per 16-column tile
//   A  : joint attention per (agent, range of cached rows, head): the 4 waves split the 32-row tiles and
//        merge in LDS; each wave keeps a ring of raw tiles in flight; the expert's own rows are tiles of
//        the agent's last range; when an agent's rows were split over several ranges, the last range to
//        finish merges them (log-sum-exp).  Units after the first are taken from a per-layer counter.
//   O  : output projection, split-K by head group; the last split of each column tile adds the
//        residual and writes h_mid plus per-tile sums of squares for the next RMSNorm
//   F1 : RMSNorm + gate/up projection with SwiGLU
//   D  : down projection, split-K; the last split adds the residual and writes h_out
// and the head pools the first T tokens at the end.  Phases are connected by per-producer flags, not
// grid barriers: a producer writes its outputs with device-coherent stores, waits for them to
// complete, and stores a flag holding a stamp that grows with (launch, layer); a consumer polls only
// the flags of the tiles it reads.
//
// Coherence.  Each XCD has its own L2, and a cache line written in parts by workgroups on different
// XCDs can sit in a reader's L2 with parts missing.  Buffers that many workgroups read (the bf16
// projection inputs, their sums of squares, the SwiGLU output, the attention output) are therefore laid
// out so that every 128-byte line has exactly one producer (tile-major: [column tile][row][16 or 8
// columns], rows padded), are written once per launch, and are read with ordinary loads after the
// producer's flag, so they are served from L2 after the first reader of an XCD.  Everything else
// produced inside the launch (queries, the expert's own keys/values, split-K partials, the residual
// stream, attention partial states) is read with device-coherent loads.  Weights and cache rows are
// read-only.  Every wait is bounded in real time; on timeout the launch records a failure and the head
// writes NaN waypoints.

#include "attn_device.h"
#include "common.h"
#include "kernels.h"

namespace fsx {

// threadIdx.x, re-read at each use through an empty asm statement.  Otherwise the compiler hoists the
// lane-dependent addresses of every phase out of the layer loop and keeps them all live at once, which
// exhausts the register file; recomputing them where they are used costs a few instructions.
__device__ __forceinline__ int tix() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

constexpr int XSTR = 520;  // LDS row stride (bf16 elements) of staged activations: 512 + 8 padding
constexpr int NTHR = 256;
constexpr int UMAX = 4;    // projection units whose weights a wave holds in registers at once
constexpr int MTMAX = 5;   // 16-row tiles per staged chunk (80 rows)
constexpr int DH = 128;    // head width of the fused path
constexpr int STW = 16 * DH + 32;  // LDS floats of one wave's attention state: O[16][128], (m, l)[16]
constexpr int NQW = 3;     // query tiles a wave carries at once in the many-query attention variant

struct TickLds {
  union {
    struct {
      uint16_t x[MTMAX * 16][XSTR];  // staged activation rows (bf16) of the current chunk
      f32x4 red[4][MTMAX][WAVE];     // cross-wave reduction of projection accumulators
    } p;
    struct {
      float st[4][STW];                // per-wave attention states
      uint16_t qs[NQW * 16][DH + 8];  // many-query attention: the unit's query tiles (bf16 or fp16)
    } a;
  } u;
  float rope[MTMAX * 16][DH / 2][2];  // rotary cos, sin of the chunk's rows
  float r[MTMAX * 16];  // RMSNorm row scales of the chunk
  float tmp[512];       // head scratch
  float red2[16][16];   // head: per-wave partial sums
  float hr[64];         // head: row scales of the pooled tokens (at most 64)
  int ok;
  int last;
  int next;
};

__device__ __forceinline__ uint64_t stamp_of(const TickArgs& a, int layer, int n_layers) {
  return a.epoch * (uint64_t)(n_layers + 2) + (uint64_t)(layer + 2);
}
__device__ __forceinline__ uint64_t fail_tag(const TickArgs& a) { return a.epoch + 1; }

// Wave-level wait until flags[(i / inner) * stride + i % inner] >= target for i < n.  Up to 256 flags are
// polled per round trip.  False on timeout or when another workgroup has already recorded a failure for
// this launch.
__device__ __forceinline__ bool wave_wait(const uint64_t* flags, int n, uint64_t target, const TickArgs& a,
                                          int inner = 1 << 30, int stride = 0) {
  constexpr int GR = 4;  // groups of 64 flags per round trip
  const int lane = tix() & 63;
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  for (int base = 0; base < n; base += GR * WAVE) {
    int64_t fi[GR];
#pragma unroll
    for (int g = 0; g < GR; ++g) {
      const int i = base + g * WAVE + lane;
      fi[g] = i < n ? (int64_t)(i / inner) * stride + i % inner : -1;
    }
    for (uint32_t spin = 0;; ++spin) {
      uint64_t v[GR];
#pragma unroll
      for (int g = 0; g < GR; ++g) v[g] = fi[g] >= 0 ? ld_dev(flags + fi[g]) : target;
      bool ok = true;
#pragma unroll
      for (int g = 0; g < GR; ++g) ok = ok && v[g] >= target;
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

__device__ __forceinline__ bool wg_wait(const uint64_t* flags, int n, uint64_t target, const TickArgs& a, TickLds& L,
                                        int inner = 1 << 30, int stride = 0) {
  if (tix() < WAVE) {
    const bool ok = wave_wait(flags, n, target, a, inner, stride);
    if (tix() == 0) L.ok = ok;
  }
  __syncthreads();
  const bool ok = L.ok;
  __syncthreads();
  return ok;
}

__device__ __forceinline__ void trace_mark(const TickArgs& a, int ev, int n_layers) {
  if (a.trace && tix() == 0)
    a.trace[(int64_t)blockIdx.x * trace_events(n_layers) + ev] = __builtin_amdgcn_s_memrealtime();
}

// sub-phase mark k (0..10) of layer l
#define TICK_SUB(l, k) trace_mark(a, 2 + 16 * (l) + 5 + (k), dm.n_layers)

// ------------------------------------------------------------------------------------------ staging
// Stage rows [m0, m0+rows) x K columns (K/8 <= 64 chunks of 16 bytes) of a bf16 activation into L.x with
// direct global->LDS loads (one instruction per row: lane l brings columns 8l..8l+7), the rotary rows into
// L.rope when given, and, when ssq is given, the RMSNorm row scales r[row] = 1/sqrt(mean(h^2) + eps) from the
// per-16-column sums of squares ssq[tile][Ms] into L.r.  TW = 0: row-major source [M][ld]; TW = 16 or 8:
// tile-major source [K/TW][ld = Mp][TW].  Every load is issued before any is waited for; ends with a
// barrier.  Rows past `rows` are left as they are: an MFMA output row depends only on its input row, and
// those rows are never stored.
template <int TW>
__device__ __forceinline__ void stage(const uint16_t* src, int ld, int m0, int rows, int K, const float* ssq, int Ms,
                                      int Kn, float eps, TickLds& L, const float* rope = nullptr) {
  const int tid = tix(), wave = tid >> 6, lane = tid & 63;
  const int cpr = K / 8;  // chunks per row
  if (lane < cpr) {
    int64_t off;  // element offset of lane's chunk in row 0 of the chunk
    if (TW == 0)
      off = (int64_t)m0 * ld + lane * 8;
    else if (TW == 16)
      off = ((int64_t)(lane >> 1) * ld + m0) * 16 + (lane & 1) * 8;
    else
      off = ((int64_t)lane * ld + m0) * 8;
    const int64_t row_step = TW == 0 ? ld : TW;  // elements between consecutive rows
    for (int m = wave; m < rows; m += 4) load_lds16(src + off + (int64_t)m * row_step, &L.u.p.x[m][0]);
  }
  if (rope) {  // rows [M][DH/2][2] floats, 512 bytes: one instruction per 2 rows
    for (int m = 2 * wave; m < rows; m += 8)
      if (m + (lane >> 5) < rows) load_lds16(rope + ((int64_t)(m0 + m) * DH + lane * 4), &L.rope[m][0][0]);
  }
  float part[MTMAX];
  const int g = tid & 15, rw = tid >> 4, ntn = Kn / 16;  // ntn <= 32
  if (ssq) {
#pragma unroll
    for (int p = 0; p < MTMAX; ++p) {
      const int i = rw + 16 * p;
      float s0 = 0.f, s1 = 0.f;
      if (i < rows) {
        if (g < ntn) s0 = ssq[(int64_t)g * Ms + m0 + i];
        if (g + 16 < ntn) s1 = ssq[(int64_t)(g + 16) * Ms + m0 + i];
      }
      part[p] = s0 + s1;
    }
#pragma unroll
    for (int p = 0; p < MTMAX; ++p) {
      float s = part[p];
      s += shfl_xor(s, 8);
      s += shfl_xor(s, 4);
      s += shfl_xor(s, 2);
      s += shfl_xor(s, 1);
      const int i = rw + 16 * p;
      if (g == 0) L.r[i] = i < rows ? 1.0f / sqrtf(s / (float)Kn + eps) : 0.f;
    }
  }
  vm_wait_all();  // the direct loads (and any weight loads issued earlier) are complete
  __syncthreads();
}

// ------------------------------------------------------------------------------------------ projections
// A projection unit is one 16-column tile over a range of nkb k-blocks; wave w owns the unit's k-blocks
// i = w, w+4, w+8, w+12 (a range is at most 512 columns = 16 blocks), whose 1 KiB weight blocks it holds
// in registers.
__device__ __forceinline__ void load_unit_w(const uint4* __restrict__ wtile, int kb0, int nkb, uint4 w[4]) {
  const int wave = tix() >> 6, lane = tix() & 63;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = wave + 4 * j;
    w[j] = i < nkb ? ld_global(wtile + (int64_t)(kb0 + i) * WAVE + lane) : make_uint4(0, 0, 0, 0);
  }
}

// acc = staged x (mt_n row tiles, k-blocks 0..nkb-1 of the unit's range) times the unit's weights, summed
// over the 4 waves through LDS and handed to epi(mt, C-layout values, c, grp) by wave mt % 4.
template <typename Epi>
__device__ __forceinline__ void unit_gemm(const uint4 w[4], int nkb, int mt_n, TickLds& L, Epi epi) {
  const int wave = tix() >> 6, lane = tix() & 63;
  const int c = lane & 15, grp = lane >> 4;
  // every row tile of the chunk buffer is multiplied (straight-line code); tiles past mt_n are not used
  f32x4 acc[MTMAX];
#pragma unroll
  for (int mt = 0; mt < MTMAX; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = wave + 4 * j;
    if (i < nkb) {
      uint4 xa[MTMAX];
#pragma unroll
      for (int mt = 0; mt < MTMAX; ++mt) xa[mt] = *reinterpret_cast<const uint4*>(&L.u.p.x[mt * 16 + c][i * 32 + 8 * grp]);
#pragma unroll
      for (int mt = 0; mt < MTMAX; ++mt) acc[mt] = mfma_bf16(xa[mt], w[j], acc[mt]);
    }
  }
#pragma unroll
  for (int mt = 0; mt < MTMAX; ++mt) L.u.p.red[wave][mt][lane] = acc[mt];
  __syncthreads();
  for (int mt = wave; mt < mt_n; mt += 4) {
    const f32x4 s = L.u.p.red[0][mt][lane] + L.u.p.red[1][mt][lane] + L.u.p.red[2][mt][lane] + L.u.p.red[3][mt][lane];
    epi(mt, s, c, grp);
  }
  __syncthreads();
}

// Last split of a column tile: h_dst[m][tile] = h_src[m][tile] + sum_s part[s][m][tile] (fixed order); the
// tile also goes to hb_dst (bf16, tile-major [tile][Mp][16]) and ssq_dst[tile][m] = sum over the tile of
// h_dst^2.  Resets the tile's counter and publishes its flag.
__device__ __forceinline__ void reduce_tile(const TickArgs& a, const TickParams& tp, const Dims& dm, int nt, int nsplit,
                                            const float* h_src, float* h_dst, uint16_t* hb_dst, float* ssq_dst,
                                            uint32_t* cnt, uint64_t* flag, uint64_t st) {
  const int M = tp.M, d = dm.d, total = M * 16;
  constexpr int BATCH = 2;
  for (int i0 = tix(); i0 < total; i0 += BATCH * NTHR) {
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
      if (idx < total && (c & 1) == 0)
        st_dev(reinterpret_cast<uint32_t*>(hb_dst + ((int64_t)nt * tp.Mp + m) * 16 + c), pack_bf16x2(v, vn));
      float sq = v * v;
      sq += shfl_xor(sq, 8);
      sq += shfl_xor(sq, 4);
      sq += shfl_xor(sq, 2);
      sq += shfl_xor(sq, 1);
      if (c == 0 && idx < total) st_dev_f(ssq_dst + (int64_t)nt * tp.Ms + m, sq);
    }
  }
  if (tix() == 0) st_dev(cnt + nt, 0u);
  stores_done();
  __syncthreads();
  if (tix() == 0) st_dev(flag + nt, st);
}

// ------------------------------------------------------------------------------------------ embed
// Units 0 .. d/16-1: column tile u of every row (h0, its bf16 tile and sums of squares); units d/16 .. d/16+M-1:
// the rotary table of row m = u - d/16 (fp64 angle).  The units also return every counter to zero.
__device__ __forceinline__ void phase_embed(const TickArgs& a, const TickParams& tp, const Dims& dm, TickLds& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, half = dm.Dh / 2, nt = d / 16;
  const uint64_t st = stamp_of(a, -1, dm.n_layers);
  const int n_units = nt + M;
  for (int u = blockIdx.x; u < n_units; u += G) {
    if (u < nt) {
      // thread: row m = i / 8, column pair 2 * (i % 8)
      for (int i = tix(); i < M * 8; i += NTHR) {
        const int m = i >> 3, cp = (i & 7) * 2, n = u * 16 + cp;
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
        st_dev(reinterpret_cast<uint32_t*>(a.hb0 + ((int64_t)u * tp.Mp + m) * 16 + cp), pack_bf16x2(v0, v1));
        float sq = v0 * v0 + v1 * v1;  // the 8 threads of a row are adjacent lanes
        sq += shfl_xor(sq, 4);
        sq += shfl_xor(sq, 2);
        sq += shfl_xor(sq, 1);
        if ((i & 7) == 0) st_dev_f(a.ssq0 + (int64_t)u * tp.Ms + m, sq);
      }
    } else {
      const int m = u - nt, b = m / tp.S, t = m % tp.S;
      for (int j = tix(); j < half; j += NTHR) {
        double cs = 1.0, sn = 0.0;
        if (dm.rope_base > 0.f) {
          const double ang = (double)(tp.pos[b] + t) * pow((double)dm.rope_base, -2.0 * (double)j / (double)dm.Dh);
          cs = cos(ang);
          sn = sin(ang);
        }
        st_dev_f(a.rope + ((int64_t)m * half + j) * 2, (float)cs);
        st_dev_f(a.rope + ((int64_t)m * half + j) * 2 + 1, (float)sn);
      }
    }
    // return the counters to zero (robust to an earlier launch that stopped midway)
    for (int i = u * NTHR + tix(); i < a.n_att_cnt; i += n_units * NTHR) st_dev(a.att_cnt + i, 0u);
    for (int i = u * NTHR + tix(); i < dm.n_layers; i += n_units * NTHR) st_dev(a.sched + i, 0u);
    if (u == 0)
      for (int i = tix(); i < nt; i += NTHR) {
        st_dev(a.o_cnt + i, 0u);
        st_dev(a.d_cnt + i, 0u);
      }
    stores_done();
    __syncthreads();
    if (tix() == 0) st_dev(a.f_embed + u, st);
  }
}

// ------------------------------------------------------------------------------------------ Q
// One wave per projection unit: the wave holds the unit's 16-column tile for every k-block (K <= 512) in
// registers and multiplies all staged row tiles, so the units of a workgroup run side by side with no
// cross-wave reduction.
__device__ __forceinline__ void load_unit_w_full(const uint4* __restrict__ wtile, int nkb, uint4 w[16]) {
  const int lane = tix() & 63;
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i] = i < nkb ? ld_global(wtile + (int64_t)i * WAVE + lane) : make_uint4(0, 0, 0, 0);
}

template <typename Epi>
__device__ __forceinline__ void wave_gemm(const uint4 w[16], int nkb, int mt_n, TickLds& L, Epi epi) {
  const int lane = tix() & 63, c = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int mt = 0; mt < MTMAX; ++mt) {
    if (mt < mt_n) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (i < nkb) acc = mfma_bf16(*reinterpret_cast<const uint4*>(&L.u.p.x[mt * 16 + c][i * 32 + 8 * grp]), w[i], acc);
      epi(mt, acc, c, grp);
    }
  }
}

__device__ __forceinline__ bool phase_qkv(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, A = dm.A, Dh = dm.Dh, half = Dh / 2;
  const int wave = tix() >> 6;
  const int n_units = 3 * A / 16;
  const TickLayer& W = a.layers[l];
  const int KB = d / 32;
  const float qs = LOG2E / sqrtf((float)Dh);
  const uint16_t* hbsrc = l == 0 ? a.hb0 : a.hbout + (int64_t)(l - 1) * tp.Mp * d;
  const float* ssq = l == 0 ? a.ssq0 : a.ssq_out + (int64_t)(l - 1) * (d / 16) * tp.Ms;
  bool waited = false;
  for (int u0 = blockIdx.x; u0 < n_units; u0 += 4 * G) {
    const int u = u0 + wave * G;  // this wave's unit in this round
    const bool mine = u < n_units;
    uint4 w[16];
    if (mine) load_unit_w_full(W.wqkv + (int64_t)u * KB * WAVE, KB, w);
    if (!waited) {
      TICK_SUB(l, 0);
      const bool ok = l == 0 ? wg_wait(a.f_embed, d / 16 + M, stamp_of(a, -1, dm.n_layers), a, L)
                             : wg_wait(a.f_hout, d / 16, stamp_of(a, l - 1, dm.n_layers), a, L);
      if (!ok) return false;
      waited = true;
      TICK_SUB(l, 1);
    }
    const int sec = (u * 16) / A;  // 0 q, 1 k, 2 v
    const int nl0 = u * 16 - sec * A;
    for (int m0 = 0; m0 < M; m0 += MTMAX * 16) {
      const int rows = min(MTMAX * 16, M - m0), mt_n = (rows + 15) / 16;
      // rotary rows ([M][Dh/2][2], 512 bytes each, one producer per row, complete before any projection
      // starts) are read with ordinary loads
      stage<16>(hbsrc, tp.Mp, m0, rows, d, ssq, tp.Ms, d, dm.eps, L, a.rope);
      TICK_SUB(l, 2);
      if (mine) {
        wave_gemm(w, KB, mt_n, L, [&](int mt, f32x4 s, int c, int grp) {
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
              const float cs = L.rope[mt * 16 + 4 * grp + i][j][0];
              const float sn = L.rope[mt * 16 + 4 * grp + i][j][1];
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
      __syncthreads();  // the next chunk overwrites the staged rows
    }
  }
  TICK_SUB(l, 3);
  stores_done();
  __syncthreads();
  TICK_SUB(l, 4);
  if (tix() == 0) {
    const uint64_t st = stamp_of(a, l, dm.n_layers);
    for (int u = blockIdx.x; u < n_units; u += G) st_dev(a.f_qkv + u, st);
  }
  return true;
}

// ------------------------------------------------------------------------------------------ A
// Raw registers of one 32-row tile, as loaded.  bf16: k[rt*4 + kb] = K row r0+16rt+c, channels 32kb+8grp..+7;
// fp8: k[rt*2 + h] = K row r0+16rt+c, channels 64h+16grp..+15 (16 bytes; the k-blocks of the score MFMA then
// hold channels 64(kb/2) + 16grp + 8(kb%2) + j, and the fp16 queries use the same order).  v[j] = V row
// r0 + (j<4 ? 4grp+j : 16+4grp+j-4), channels 8c..8c+7.  fp8 tiles hold the codes and are decoded only when
// the tile is used, so the loads of the following tiles stay in flight meanwhile.
template <int KT>
struct RawTile;
template <>
struct RawTile<0> {
  uint4 k[8];
  uint4 v[8];
};
template <>
struct RawTile<1> {
  uint4 k[4];
  uint2 v[8];
};

// Cache tile at ring rows [r0, r0+32) of a (agent, layer, head) slab; rows at or past i1 load row i0 (they are
// masked out of the softmax).
template <int KT>
__device__ __forceinline__ void load_cache_tile(const char* kb, const char* vb, int64_t start, int64_t cap, int i0,
                                                int r0, int i1, RawTile<KT>& t) {
  constexpr int ES = KT == 0 ? 2 : 1;
  constexpr int64_t RB = DH * ES;
  const int lane = tix() & 63, c = lane & 15, grp = lane >> 4;
  auto roff = [&](int i) -> int64_t {
    int64_t slot = start + (i < i1 ? i : i0);
    if (slot >= cap) slot -= cap;
    return slot * RB;
  };
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const char* p = kb + roff(r0 + 16 * rt + c);
    if constexpr (KT == 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k) t.k[rt * 4 + k] = *reinterpret_cast<const uint4*>(p + (32 * k + 8 * grp) * 2);
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) t.k[rt * 2 + h] = *reinterpret_cast<const uint4*>(p + 64 * h + 16 * grp);
    }
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int rr = r0 + (j < 4 ? 4 * grp + j : 16 + 4 * grp + (j - 4));
    const char* p = vb + roff(rr) + 8 * c * ES;
    if constexpr (KT == 0)
      t.v[j] = *reinterpret_cast<const uint4*>(p);
    else
      t.v[j] = *reinterpret_cast<const uint2*>(p);
  }
}

// Own-row tile (the expert's rows [r0, r0+32) of S, bf16, produced in this launch): device-coherent loads.
__device__ __forceinline__ void load_own_tile(const char* ks, const char* vs, int64_t srow, int r0, int S,
                                              RawTile<0>& t) {
  const int lane = tix() & 63, c = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int i = r0 + 16 * rt + c;
    const char* p = ks + (int64_t)(i < S ? i : 0) * srow;
#pragma unroll
    for (int k = 0; k < 4; ++k) t.k[rt * 4 + k] = ld_dev16(p + (32 * k + 8 * grp) * 2);
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int rr = r0 + (j < 4 ? 4 * grp + j : 16 + 4 * grp + (j - 4));
    t.v[j] = ld_dev16(vs + (int64_t)(rr < S ? rr : 0) * srow + 8 * c * 2);
  }
}

// Query fragments of query tiles tt0 .. tt0+nq-1 of agent b, head h (16 queries x 128 channels each, B operand
// of S^T = K Q^T): bf16 in plain channel order (F16 = false), or fp16 in the channel order of fp8 key tiles.
template <int NQ, bool F16>
__device__ __forceinline__ void load_q(const TickArgs& a, const TickParams& tp, const Dims& dm, int b, int h, int tt0,
                                       int nq, uint4 (&q)[NQ][4]) {
  const int lane = tix() & 63, grp = lane >> 4;
#pragma unroll
  for (int tt = 0; tt < NQ; ++tt) {
    const int t = (tt0 + tt) * 16 + (lane & 15);
    const bool tv = tt < nq && t < tp.S;
    const float* row = a.q + ((int64_t)b * tp.S + (tv ? t : 0)) * dm.A + (int64_t)h * DH;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
      const int ch = F16 ? 64 * (kb >> 1) + 16 * grp + 8 * (kb & 1) : 32 * kb + 8 * grp;
      if (tv) {
        lo = ld_dev_f4(row + ch);
        hi = ld_dev_f4(row + ch + 4);
      }
      if (F16)
        q[tt][kb] = make_uint4(pack_f16x2(lo.x, lo.y), pack_f16x2(lo.z, lo.w), pack_f16x2(hi.x, hi.y),
                               pack_f16x2(hi.z, hi.w));
      else
        q[tt][kb] = make_uint4(pack_bf16x2(lo.x, lo.y), pack_bf16x2(lo.z, lo.w), pack_bf16x2(hi.x, hi.y),
                               pack_bf16x2(hi.z, hi.w));
    }
  }
}

// The unit's query tiles tt0 .. tt0+nq-1 into LDS rows (16 per tile) of 128 channels, bf16 or fp16; ends
// with a barrier.
template <bool F16>
__device__ __forceinline__ void load_q_lds(const TickArgs& a, const TickParams& tp, const Dims& dm, int b, int h,
                                           int tt0, int nq, TickLds& L) {
  for (int i = tix(); i < nq * 16 * (DH / 8); i += NTHR) {
    const int row = i / (DH / 8), c8 = (i % (DH / 8)) * 8;
    const int t = tt0 * 16 + row;
    float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
    if (t < tp.S) {
      const float* src = a.q + ((int64_t)b * tp.S + t) * dm.A + (int64_t)h * DH + c8;
      lo = ld_dev_f4(src);
      hi = ld_dev_f4(src + 4);
    }
    uint4 v;
    if (F16)
      v = make_uint4(pack_f16x2(lo.x, lo.y), pack_f16x2(lo.z, lo.w), pack_f16x2(hi.x, hi.y), pack_f16x2(hi.z, hi.w));
    else
      v = make_uint4(pack_bf16x2(lo.x, lo.y), pack_bf16x2(lo.z, lo.w), pack_bf16x2(hi.x, hi.y), pack_bf16x2(hi.z, hi.w));
    *reinterpret_cast<uint4*>(&L.u.a.qs[row][c8]) = v;
  }
  __syncthreads();
}

// Online-softmax update of the states of the nq query tiles with one tile whose rows r0.. (valid below i1)
// are in t; qf(tt, kb) returns the B-operand fragment kb of query tile tt.  fp8 tiles (KT 1) are decoded to
// fp16 (exact) and use fp16 MFMA; their key scale multiplies the fp32 scores (the value scale is applied to
// the output once, after the cache tiles).  The running max of a query only moves when a score exceeds it
// by more than 2^8 (log2 units), so the accumulators are rescaled rarely; probabilities stay below 2^8.
constexpr float RESCALE_LOG2 = 8.0f;
template <int KT, int NQ, typename QF>
__device__ __forceinline__ void tile_compute(const RawTile<KT>& t, QF qf, int nq, int r0, int i1, float kscale,
                                             f32x4 (&o)[NQ][8], float (&m_run)[NQ], float (&l_run)[NQ]) {
  constexpr bool F16 = KT == 1;
  const int lane = tix() & 63, grp = lane >> 4;
  uint4 kf[8], vr[8];
  if constexpr (KT == 0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      kf[i] = t.k[i];
      vr[i] = t.v[i];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      kf[2 * i] = make_uint4(e4m3x2_to_f16x2(t.k[i].x, false), e4m3x2_to_f16x2(t.k[i].x, true),
                             e4m3x2_to_f16x2(t.k[i].y, false), e4m3x2_to_f16x2(t.k[i].y, true));
      kf[2 * i + 1] = make_uint4(e4m3x2_to_f16x2(t.k[i].z, false), e4m3x2_to_f16x2(t.k[i].z, true),
                                 e4m3x2_to_f16x2(t.k[i].w, false), e4m3x2_to_f16x2(t.k[i].w, true));
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
      vr[i] = make_uint4(e4m3x2_to_f16x2(t.v[i].x, false), e4m3x2_to_f16x2(t.v[i].x, true),
                         e4m3x2_to_f16x2(t.v[i].y, false), e4m3x2_to_f16x2(t.v[i].y, true));
  }
  uint4 vt[8];
  transpose8x8_b16(vr, vt);
#pragma unroll
  for (int tt = 0; tt < NQ; ++tt) {
    if (tt < nq) {
      f32x4 s[2];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        s[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint4 qk = qf(tt, k);
          s[rt] = F16 ? mfma_f16(kf[rt * 4 + k], qk, s[rt]) : mfma_bf16(kf[rt * 4 + k], qk, s[rt]);
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int rr = r0 + 16 * rt + 4 * grp + i;
          const float v = rr < i1 ? (KT == 1 ? s[rt][i] * kscale : s[rt][i]) : -INFINITY;
          s[rt][i] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, shfl_xor(mx, 16));
      mx = fmaxf(mx, shfl_xor(mx, 32));
      const bool grow = mx > m_run[tt] + RESCALE_LOG2;
      if (__any(grow)) {
        const float m_new = grow ? mx : m_run[tt];
        const float alpha = exp2f(m_run[tt] - m_new);
        l_run[tt] *= alpha;
        m_run[tt] = m_new;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float a_i = shfl(alpha, 4 * grp + i);
#pragma unroll
          for (int k = 0; k < 8; ++k) o[tt][k][i] *= a_i;
        }
      }
      float p[8], ps = 0.f;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          p[rt * 4 + i] = exp2f(s[rt][i] - m_run[tt]);
          ps += p[rt * 4 + i];
        }
      l_run[tt] += ps;
      uint4 pf;
      if (F16)
        pf = make_uint4(pack_f16x2(p[0], p[1]), pack_f16x2(p[2], p[3]), pack_f16x2(p[4], p[5]), pack_f16x2(p[6], p[7]));
      else
        pf = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                        pack_bf16x2(p[6], p[7]));
#pragma unroll
      for (int k = 0; k < 8; ++k) o[tt][k] = F16 ? mfma_f16(pf, vt[k], o[tt][k]) : mfma_bf16(pf, vt[k], o[tt][k]);
    }
  }
}

// write a wave's state (o in the PV C layout, m and the lane-partial l) to LDS slot w
__device__ __forceinline__ void state_to_lds(float* stw, const f32x4 o[8], float m_run, float l_run) {
  const int lane = tix() & 63, c = lane & 15, grp = lane >> 4;
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

// Merge the 4 waves' LDS states of query tile tt: each thread owns (t, 8 channels).  If final, normalise into
// the attention output; else store the unnormalised partial of slot `item`.
__device__ __forceinline__ void merge_states(const TickArgs& a, const TickParams& tp, const Dims& dm, int l,
                                             const AUnit& U, int tt, bool final_out, int64_t item, TickLds& L) {
  const int t = tix() >> 4, d0 = (tix() & 15) * 8;
  float Mx = -INFINITY;
#pragma unroll
  for (int w = 0; w < 4; ++w) Mx = fmaxf(Mx, L.u.a.st[w][2048 + 2 * t]);
  float Ls = 0.f, acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float* stw = L.u.a.st[w];
    const float f = Mx == -INFINITY ? 0.f : exp2f(stw[2048 + 2 * t] - Mx);
    Ls += stw[2048 + 2 * t + 1] * f;
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += stw[t * 128 + d0 + k] * f;
  }
  if (final_out) {
    const int tok = tt * 16 + t;
    if (tok < tp.S) {
      const float inv = 1.0f / Ls;
      uint16_t* dst = a.attn + (int64_t)l * tp.M * dm.A + ((int64_t)U.b * tp.S + tok) * dm.A + (int64_t)U.h * DH + d0;
      st_dev16(dst, make_uint4(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                               pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)));
    }
  } else {
    float* po = a.att_o + (item * 16 + t) * 128 + d0;
    st_dev_f4(po, make_float4(acc[0], acc[1], acc[2], acc[3]));
    st_dev_f4(po + 4, make_float4(acc[4], acc[5], acc[6], acc[7]));
    if ((tix() & 15) == 0) {
      st_dev_f(a.att_ml + item * 32 + 2 * t, Mx);
      st_dev_f(a.att_ml + item * 32 + 2 * t + 1, Ls);
    }
  }
}

// the last range of an agent to finish merges the partials of all its ranges (fixed order)
__device__ __forceinline__ void combine_ranges(const TickArgs& a, const TickParams& tp, const Dims& dm, int l,
                                               const AUnit& U) {
  const int t = tix() >> 4, d0 = (tix() & 15) * 8;
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
      uint16_t* dst = a.attn + (int64_t)l * tp.M * dm.A + ((int64_t)U.b * tp.S + tok) * dm.A + (int64_t)U.h * DH + d0;
      st_dev16(dst, make_uint4(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                               pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)));
    }
  }
}

// The tiles of one unit for query tiles tt0 .. tt0+nq-1 (nq <= NQ): wave w takes cache tiles w, w+4, ..., kept
// PD deep in registers, then the own-row tiles that continue the same round robin; the states are merged
// through LDS and written out.  One query tile is held in registers; several are read from LDS.  Returns
// false if a wait failed.
template <int KT, int NQ, int PD>
__device__ __forceinline__ bool attn_unit(const TickArgs& a, const TickParams& tp, const Dims& dm, int l,
                                          const AUnit& U, int tt0, int nq, TickLds& L) {
  const int wave = tix() >> 6, lane = tix() & 63, c16 = lane & 15, grp = lane >> 4;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  // this wave's cache tiles: j = wave + 4 i, i < nc
  const int nc = U.nct > wave ? (U.nct - wave + 3) / 4 : 0;
  RawTile<KT> ring[PD];
  auto cache_tile = [&](int i, RawTile<KT>& t) {
    const int ii = i < nc ? i : nc - 1;
    load_cache_tile<KT>(U.kc, U.vc, tp.start[U.b], a.cv.cap, U.i0, U.i0 + 32 * (wave + 4 * ii), U.i1, t);
  };
  // the first tiles do not depend on this layer's projections: issue them before waiting
  if (nc > 0) {
#pragma unroll
    for (int dd = 0; dd < PD; ++dd) cache_tile(dd, ring[dd]);
  }
  {
    // the q, k and v column tiles of this head
    const bool ok = wave_wait(a.f_qkv + U.h * (DH / 16), 3 * (DH / 16), st, a, DH / 16, dm.A / 16);
    if (!ok && lane == 0) L.ok = 0;
    __syncthreads();
    if (!L.ok) return false;
  }
  f32x4 o[NQ][8];
  float m_run[NQ], l_run[NQ];
#pragma unroll
  for (int tt = 0; tt < NQ; ++tt) {
#pragma unroll
    for (int k = 0; k < 8; ++k) o[tt][k] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[tt] = -INFINITY;
    l_run[tt] = 0.f;
  }
  uint4 qr[4];  // NQ == 1: the query fragments
  if (NQ == 1)
    load_q<1, KT == 1>(a, tp, dm, U.b, U.h, tt0, nq, reinterpret_cast<uint4(&)[1][4]>(qr));
  else
    load_q_lds<KT == 1>(a, tp, dm, U.b, U.h, tt0, nq, L);
  // LDS queries are in plain channel order; fp8 key tiles want the permuted order (see RawTile)
  auto qf = [&](int tt, int k) -> uint4 {
    if (NQ == 1) return qr[k];
    const int ch = KT == 1 ? 64 * (k >> 1) + 16 * grp + 8 * (k & 1) : 32 * k + 8 * grp;
    return *reinterpret_cast<const uint4*>(&L.u.a.qs[tt * 16 + c16][ch]);
  };
  auto qf_own = [&](int tt, int k) -> uint4 {
    if (NQ == 1) return qr[k];
    return *reinterpret_cast<const uint4*>(&L.u.a.qs[tt * 16 + c16][32 * k + 8 * grp]);
  };
  int i = 0;
  for (; i + PD <= nc; i += PD) {
#pragma unroll
    for (int dd = 0; dd < PD; ++dd) {
      tile_compute<KT, NQ>(ring[dd], qf, nq, U.i0 + 32 * (wave + 4 * (i + dd)), U.i1, U.ksc, o, m_run, l_run);
      cache_tile(i + dd + PD, ring[dd]);
    }
  }
#pragma unroll
  for (int dd = 0; dd < PD; ++dd)
    if (i + dd < nc)
      tile_compute<KT, NQ>(ring[dd], qf, nq, U.i0 + 32 * (wave + 4 * (i + dd)), U.i1, U.ksc, o, m_run, l_run);
  if (KT == 1) {
    // fp8 values carry their scale: apply it to the cache part of the output before the own rows join
#pragma unroll
    for (int tt = 0; tt < NQ; ++tt)
#pragma unroll
      for (int k = 0; k < 8; ++k) o[tt][k] *= U.vsc;
  }
  // own rows (bf16): tiles U.nct .. U.nct+nst-1 of the round robin
  if (U.nst > 0) {
    if (KT == 1) {  // the queries again, as bf16
      if (NQ == 1) {
        load_q<1, false>(a, tp, dm, U.b, U.h, tt0, nq, reinterpret_cast<uint4(&)[1][4]>(qr));
      } else {
        __syncthreads();  // every wave is done with the fp16 queries
        load_q_lds<false>(a, tp, dm, U.b, U.h, tt0, nq, L);
      }
    }
    const int first_own = (wave - U.nct % 4 + 4) % 4;
    for (int j = first_own; j < U.nst; j += 4) {
      RawTile<0> t;
      load_own_tile(U.ks, U.vs, (int64_t)dm.A * 2, 32 * j, tp.S, t);
      tile_compute<0, NQ>(t, qf_own, nq, 32 * j, tp.S, 1.f, o, m_run, l_run);
    }
  }
  const bool final_out = U.nr == 1;
  const int64_t pair = (int64_t)(tp.range_prefix[U.b] + U.r) * dm.H + U.h;
#pragma unroll
  for (int tt = 0; tt < NQ; ++tt) {
    if (tt < nq) {
      state_to_lds(L.u.a.st[wave], o[tt], m_run[tt], l_run[tt]);
      __syncthreads();
      merge_states(a, tp, dm, l, U, tt0 + tt, final_out, pair * tp.n_tt + tt0 + tt, L);
      __syncthreads();
    }
  }
  return true;
}

// Attention units are (agent, range, head), numbered agent by agent in the planner's order (largest ranges
// first), heads fastest.  Workgroup w starts with unit w; further units come from a per-layer counter.
template <int KT>
__device__ __forceinline__ bool phase_attn(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  constexpr int ES = KT == 0 ? 2 : 1;
  const int G = gridDim.x;
  const int H = dm.H, A = dm.A, n_tt = tp.n_tt;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const int n_units = tp.n_units;
  int u = blockIdx.x;
  bool first = true;
  while (u < n_units) {
    // take the next unit now; the answer is needed only at the end of this one
    uint32_t nxt = 0;
    if (tix() == 0) nxt = atomic_add_dev(a.sched + l, 1u);
    AUnit U;
    int k = 0;
    while (k + 1 < tp.B && tp.unit_prefix[k + 1] <= u) ++k;
    const int b = tp.order[k];
    const int rem = u - tp.unit_prefix[k];
    U.b = b;
    U.r = rem / H;
    U.h = rem - U.r * H;
    U.nr = tp.range_prefix[b + 1] - tp.range_prefix[b];
    U.i0 = U.r * tp.range_rows[b];
    U.i1 = min(U.i0 + tp.range_rows[b], tp.len[b]);
    U.nct = U.i1 > U.i0 ? (U.i1 - U.i0 + 31) / 32 : 0;
    U.nst = U.r == U.nr - 1 ? (tp.S + 31) / 32 : 0;
    const int64_t slab = (((int64_t)b * a.cv.n_layers + l) * H + U.h) * a.cv.cap;  // head-major (b, l, h) ring
    U.kc = (const char*)a.cv.k + slab * DH * ES;
    U.vc = (const char*)a.cv.v + slab * DH * ES;
    U.ks = (const char*)a.kself + ((int64_t)b * tp.S * A + (int64_t)U.h * DH) * 2;
    U.vs = (const char*)a.vself + ((int64_t)b * tp.S * A + (int64_t)U.h * DH) * 2;
    U.ksc = U.vsc = 1.f;
    if (KT == 1) {
      const int64_t si = ((int64_t)b * a.cv.n_layers + l) * H + U.h;
      U.ksc = a.cv.k_scale[si];
      U.vsc = a.cv.v_scale[si];
    }
    bool ok = true;
    if (n_tt == 1) {
      ok = attn_unit<KT, 1, KT == 0 ? 3 : 4>(a, tp, dm, l, U, 0, 1, L);
    } else {
      for (int tt0 = 0; tt0 < n_tt && ok; tt0 += NQW)
        ok = attn_unit<KT, NQW, 2>(a, tp, dm, l, U, tt0, min(NQW, n_tt - tt0), L);
    }
    if (!ok) return false;
    if (first) TICK_SUB(l, 5);
    if (tix() == 0) L.next = G + (int)nxt;
    stores_done();
    __syncthreads();
    if (first) TICK_SUB(l, 6);
    const int ci = b * H + U.h;
    // an (agent, head) is complete when all its ranges are written
    const uint32_t need = (uint32_t)U.nr;
    if (tix() == 0) L.last = need == 1 ? 1 : atomic_add_dev(a.att_cnt + ci, 1u) == need - 1;
    __syncthreads();
    if (L.last) {
      if (need > 1) combine_ranges(a, tp, dm, l, U);
      if (tix() == 0 && need > 1) st_dev(a.att_cnt + ci, 0u);
      stores_done();
      __syncthreads();
      if (tix() == 0) st_dev(a.f_attn + ci, st);
    }
    u = L.next;
    first = false;
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------------------------------ O
__device__ __forceinline__ bool phase_oproj(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
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
    for (int m0 = 0; m0 < M; m0 += MTMAX * 16) {
      const int rows = min(MTMAX * 16, M - m0), mt_n = (rows + 15) / 16;
      stage<0>(attn + ks * nk, A, m0, rows, nk, nullptr, 0, 0, 0.f, L);
      unit_gemm(w, nkb, mt_n, L, [&](int mt, f32x4 s, int c, int grp) {
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
    if (tix() == 0) L.last = atomic_add_dev(a.o_cnt + nt, 1u) == (uint32_t)(a.ks_o - 1);
    __syncthreads();
    if (u == (int)blockIdx.x) TICK_SUB(l, 9);
    if (L.last)
      reduce_tile(a, tp, dm, nt, a.ks_o, hin, a.hmid + (int64_t)l * M * d, a.hbmid + (int64_t)l * tp.Mp * d,
                  a.ssq_mid + (int64_t)l * (d / 16) * tp.Ms, a.o_cnt, a.f_hmid, st);
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------------------------------ F1
__device__ __forceinline__ bool phase_gateup(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M;
  const int n_units = 2 * dm.F / 16;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const TickLayer& W = a.layers[l];
  const uint16_t* hbmid = a.hbmid + (int64_t)l * tp.Mp * d;
  const float* ssq = a.ssq_mid + (int64_t)l * (d / 16) * tp.Ms;
  uint16_t* z = a.z + (int64_t)l * tp.Mp * dm.F;  // tile-major [F/8][Mp][8]
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
    for (int m0 = 0; m0 < M; m0 += MTMAX * 16) {
      const int rows = min(MTMAX * 16, M - m0), mt_n = (rows + 15) / 16;
      stage<16>(hbmid, tp.Mp, m0, rows, d, ssq, tp.Ms, d, dm.eps, L);
#pragma unroll
      for (int k = 0; k < UMAX; ++k) {
        const int u = u0 + k * G;
        if (u >= n_units) break;
        unit_gemm(w[k], KB, mt_n, L, [&](int mt, f32x4 s, int c, int grp) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            s[i] *= L.r[mt * 16 + 4 * grp + i];  // RMSNorm row scale
            const float up = shfl_xor(s[i], 8);
            const float gt = s[i];
            const float zz = gt / (1.0f + expf(-gt)) * up;
            const float zn = shfl_xor(zz, 1);
            const int row = m0 + mt * 16 + 4 * grp + i;
            if (c < 8 && (c & 1) == 0 && row < M)
              st_dev(reinterpret_cast<uint32_t*>(z + ((int64_t)u * tp.Mp + row) * 8 + c), pack_bf16x2(zz, zn));
          }
        });
      }
    }
  }
  stores_done();
  __syncthreads();
  if (tix() == 0)
    for (int u = blockIdx.x; u < n_units; u += G) st_dev(a.f_z + u, st);
  return true;
}

// ------------------------------------------------------------------------------------------ D
__device__ __forceinline__ bool phase_down(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, F = dm.F;
  const int ntiles = d / 16, n_units = ntiles * a.ks_d, nk = F / a.ks_d, nkb = nk / 32;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const TickLayer& W = a.layers[l];
  const uint16_t* z = a.z + (int64_t)l * tp.Mp * F;
  const float* hmid = a.hmid + (int64_t)l * M * d;
  for (int u = blockIdx.x; u < n_units; u += G) {
    const int nt = u % ntiles, ks = u / ntiles;
    uint4 w[4];
    load_unit_w(W.wd + (int64_t)nt * (F / 32) * WAVE, ks * nkb, nkb, w);
    if (!wg_wait(a.f_z + ks * nk / 8, nk / 8, st, a, L)) return false;
    for (int m0 = 0; m0 < M; m0 += MTMAX * 16) {
      const int rows = min(MTMAX * 16, M - m0), mt_n = (rows + 15) / 16;
      stage<8>(z + (int64_t)(ks * nk / 8) * tp.Mp * 8, tp.Mp, m0, rows, nk, nullptr, 0, 0, 0.f, L);
      unit_gemm(w, nkb, mt_n, L, [&](int mt, f32x4 s, int c, int grp) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = m0 + mt * 16 + 4 * grp + i;
          if (row < M) st_dev_f(a.part + ((int64_t)ks * M + row) * d + nt * 16 + c, s[i]);
        }
      });
    }
    stores_done();
    __syncthreads();
    if (tix() == 0) L.last = atomic_add_dev(a.d_cnt + nt, 1u) == (uint32_t)(a.ks_d - 1);
    __syncthreads();
    if (L.last)
      reduce_tile(a, tp, dm, nt, a.ks_d, hmid, a.hout + (int64_t)l * M * d, a.hbout + (int64_t)l * tp.Mp * d,
                  a.ssq_out + (int64_t)l * (d / 16) * tp.Ms, a.d_cnt, a.f_hout, st);
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------------------------------ head
// wp[b] = mean over t < T of RMSNorm(h[b][t]) * g_final, times W_head^T.  Thread tid owns columns tid and
// tid + 256 and holds the pooled rows in registers (16 rows per pass).
__device__ __forceinline__ void phase_head(const TickArgs& a, const TickParams& tp, const Dims& dm, bool ok, TickLds& L) {
  const int G = gridDim.x, d = dm.d, M = tp.M, nl = dm.n_layers, T = tp.T;
  const int tid = tix(), wave = tid >> 6, lane = tid & 63;
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
template <int KT>
__global__ __launch_bounds__(NTHR, 1) void k_tick(TickArgs a, TickParams tp, Dims dm) {
  __shared__ TickLds L;
  const int nl = dm.n_layers;
  trace_mark(a, 0, nl);
  if (tix() == 0) L.ok = 1;
  __syncthreads();
  phase_embed(a, tp, dm, L);
  trace_mark(a, 1, nl);
  bool ok = true;
  for (int l = 0; l < nl && ok; ++l) {
    ok = phase_qkv(a, tp, dm, l, L);
    trace_mark(a, 2 + 16 * l, nl);
    ok = ok && phase_attn<KT>(a, tp, dm, l, L);
    trace_mark(a, 3 + 16 * l, nl);
    ok = ok && phase_oproj(a, tp, dm, l, L);
    trace_mark(a, 4 + 16 * l, nl);
    ok = ok && phase_gateup(a, tp, dm, l, L);
    trace_mark(a, 5 + 16 * l, nl);
    ok = ok && phase_down(a, tp, dm, l, L);
    trace_mark(a, 6 + 16 * l, nl);
  }
  phase_head(a, tp, dm, ok, L);
  trace_mark(a, 2 + 16 * nl, nl);
}

hipError_t tick_occupancy(int kt, int* blocks_per_cu) {
  const void* f = kt == 0 ? (const void*)k_tick<0> : (const void*)k_tick<1>;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, f, NTHR, 0);
}

hipError_t launch_tick(const TickArgs& a, const TickParams& tp, const Dims& dm, int grid, hipStream_t s) {
  void* args[] = {(void*)&a, (void*)&tp, (void*)&dm};
  const void* f = a.cv.dtype == FSX_FP8_E4M3 ? (const void*)k_tick<1> : (const void*)k_tick<0>;
  return hipLaunchCooperativeKernel(f, dim3(grid), dim3(NTHR), args, 0, s);
}

}  // namespace fsx
