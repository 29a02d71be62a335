// The whole expert tick (Sec. 3.1, Eq. (1)) as ONE persistent cooperative launch, with every layer split
// over the chip's XCDs the way a tensor-parallel transformer layer is split over devices.
//
// MI355X has 8 XCDs of 32 CUs; each XCD has its own L2.  A hand-off between two workgroups of one XCD
// goes through that L2 (a flag written with a plain store and polled with a device-scope load is seen
// after ~0.3 us); a hand-off between XCDs has to go through memory (~0.55 us one way).  So XCD X owns a
// contiguous range of heads and a contiguous range of FFN columns, and a layer runs as
//   Q  : RMSNorm + q/k/v projection (+ rotary, q pre-scale) of X's heads, per 16-column tile
//   A  : joint attention of X's heads (agent, range of cached rows, head); an agent's last range merges the
//        others (log-sum-exp)
//   O  : output projection restricted to X's heads: a partial sum over X's attention columns for each
//        16-column tile of the residual
//   R1 : reduction across XCDs: column tile i of the residual belongs to one XCD, whose workgroups each
//        take a block of its rows (a piece), read the 8 partials of the piece (stamped words, polled
//        directly), add them in a fixed order to the residual and publish the piece's bf16 values and
//        sums of squares to every XCD
//   F1 : RMSNorm + gate/up projection with SwiGLU for X's FFN columns
//   D  : down projection restricted to X's FFN columns (partials)
//   R2 : reduction across XCDs as R1, giving the layer output
// All exchanges except R1 and R2 (and the residual they publish) stay inside an XCD.  Each residual element
// is reduced once, in a fixed order, so every XCD reads the same values.  The head pools the first T tokens at
// the end.
//
// Placement.  Each workgroup reads its hardware XCD id at the start of the tick and publishes it; from the
// published ids every workgroup derives its XCD rank X, its slot s among that XCD's n workgroups, and the
// number NX of XCDs, so the split is right whatever the hardware placement is.
//
// Coherence.  Inside an XCD: plain stores, a wait for them (stores_done), then a flag; readers poll flags
// and read data with device-scope loads, which are served by the XCD's L2 and never by a stale L1 line.
// Across XCDs: 8-byte words holding a 32-bit payload and a 32-bit stamp, written with device-scope stores
// and read with device-scope loads; a word is valid when its stamp is the expected one, so no flag is
// needed.  Weights and cache rows are read-only and use ordinary loads.  Every wait is bounded in real time;
// on timeout the launch records a failure and the head writes NaN waypoints.

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
constexpr int MTMAX = 5;   // 16-row tiles per staged chunk (80 rows)
constexpr int DH = 128;    // head width of the fused path
constexpr int STW = 16 * DH + 32;  // LDS floats of one wave's attention state: O[16][128], (m, l)[16]
constexpr int NQW = 6;     // many-query attention: query tiles per pass over the cache (96 queries)
constexpr int RSLOTS = 4;     // attention: LDS ring slots per wave
constexpr int RSLOT = 8192;   // bytes of one slot: an fp8 tile (32 rows) or half a bf16 tile (16 rows), K then V
constexpr int NSEG = FSX_MAX_BATCH * 4;  // attention segments (agent, local head) of one XCD, at most

// A value read from LDS that is the same in every lane, moved to a scalar register.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
// Row blocks of MTMAX * 16 rows: the projections stage and multiply one block of the M rows at a time.
__device__ __forceinline__ int row_blocks(int M) { return (M + MTMAX * 16 - 1) / (MTMAX * 16); }

struct TickLds {
  union {
    struct {
      uint16_t x[MTMAX * 16][XSTR];    // staged activation rows (bf16) of the current chunk
      f32x4 red[4][MTMAX][WAVE];       // cross-wave reduction of projection accumulators
      float rq[4][MTMAX * 16][8][2];   // q/k projection: each wave's rotary slice (cos, sin of its 8 pairs) per row
    } p;
    struct {
      // attention: each wave's cache tiles, staged by direct loads; after its last tile a wave's state goes to the
      // start of its own slots (STW floats)
      uint8_t ring[4][RSLOTS][RSLOT];
    } a;
  } u;
  alignas(16) float r[MTMAX * 16];  // RMSNorm row scales of the chunk
  float tmp[512];       // head scratch
  float red2[16][16];   // head: per-wave partial sums
  float hr[64];         // head: row scales of the pooled tokens (at most 64)
  int ok;
  int X, s, n, NX, n0;  // XCD rank, slot in the XCD, workgroups of the XCD, XCDs, workgroups of XCD 0
  // attention plan of the workgroup's XCD, made once per launch: segment g = j * B + k (local head j, agent
  // order[k]) has its tiles at work units [seg0[g], seg0[g] + segw[g]); they meet np[g] slices, the first being slice
  // sf[g], and when np[g] > 1 its partial states occupy slots pb[g] .. pb[g] + np[g] - 1 of the XCD.  amode: 1 =
  // slice s is segment s, 0 = slices of equal work; ant: work units in total
  int seg0[NSEG];
  int segw[NSEG];
  int pb[NSEG];
  int16_t sf[NSEG], np[NSEG];
  int amode, ant;
};

__device__ __forceinline__ uint64_t stamp_of(const TickArgs& a, int layer, int n_layers) {
  return a.epoch * (uint64_t)(n_layers + 2) + (uint64_t)(layer + 2);
}
__device__ __forceinline__ uint64_t fail_tag(const TickArgs& a) { return a.epoch + 1; }

// Checked inside wait loops every few spins: the elapsed real time every 4 spins, the launch's failure word (a
// device-scope vector load) every 64.
__device__ __forceinline__ bool timed_out(const TickArgs& a, uint64_t t0, uint32_t spin) {
  if ((spin & 3) != 3) return false;
  if (__builtin_amdgcn_s_memrealtime() - t0 > a.timeout_ticks) return true;
  return (spin & 63) == 63 && ld_dev(a.status) == fail_tag(a);
}

// Wave-level wait until flags[((i / inner) * stride + i % inner) * FPAD] >= target for i < n, with device-scope
// vector loads (served by the XCD's L2 for flags written inside the XCD); up to 256 flags per round trip.  False
// on timeout or when another workgroup has already recorded a failure for this launch.
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
      fi[g] = i < n ? ((int64_t)(i / inner) * stride + i % inner) * FPAD : -1;
    }
    for (uint32_t spin = 0;; ++spin) {
      // every group's loads issued, unconditionally, before any is checked: lanes past the end load flag 0 and ignore
      // it (a load behind a branch, or selected against a constant, is waited for where the branches join, which
      // made each group of a poll one more memory round trip)
      uint64_t v[GR];
#pragma unroll
      for (int g = 0; g < GR; ++g) v[g] = ld_dev(flags + (fi[g] >= 0 ? fi[g] : 0));
      bool ok = true;
#pragma unroll
      for (int g = 0; g < GR; ++g) ok = ok && (fi[g] < 0 || v[g] >= target);
      if (__all(ok)) break;
      __builtin_amdgcn_s_sleep(1);
      if (timed_out(a, t0, spin)) {
        if (lane == 0) st_dev(a.status, fail_tag(a));
        return false;
      }
    }
  }
  return true;
}

// Workgroup-level wait: wave `pw` polls, the others wait at a barrier.  Loads return in issue order, so the polling
// wave should have no long loads in flight.
__device__ __forceinline__ bool wg_wait(const uint64_t* flags, int n, uint64_t target, const TickArgs& a, TickLds& L,
                                        int inner = 1 << 30, int stride = 0, int pw = 0) {
  if ((tix() >> 6) == pw) {
    const bool ok = wave_wait(flags, n, target, a, inner, stride);
    if ((tix() & 63) == 0) L.ok = ok;
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

// ------------------------------------------------------------------------------------------ weights
// Packed weights of layer l: [W_q; W_k; W_v] (3A x d), W_o (d x A), [W_gate; W_up] (2F x d), W_down (d x F), stored
// back to back for every layer, so their addresses follow from the layer index without a memory access.
struct LayerW {
  const uint4* wqkv;
  const uint4* wo;
  const uint4* wgu;
  const uint4* wd;
};
__device__ __forceinline__ LayerW layer_w(const TickArgs& a, const Dims& dm, int l) {
  const int64_t ad = (int64_t)dm.A * dm.d * 2, fd = (int64_t)dm.F * dm.d * 2;  // bytes of one A x d / F x d matrix
  const char* base = a.wbase + (int64_t)l * (4 * ad + 3 * fd);
  LayerW w;
  w.wqkv = reinterpret_cast<const uint4*>(base);
  w.wo = reinterpret_cast<const uint4*>(base + 3 * ad);
  w.wgu = reinterpret_cast<const uint4*>(base + 4 * ad);
  w.wd = reinterpret_cast<const uint4*>(base + 4 * ad + 2 * fd);
  return w;
}

// ------------------------------------------------------------------------------------------ work split
// Heads [h0, h1) and FFN columns [f0, f1) (multiples of 32) of XCD rank X.
__device__ __forceinline__ int head_lo(int X, int NX, int H) { return X * H / NX; }
__device__ __forceinline__ int ffn_lo(int X, int NX, int F) { return 32 * (X * (F / 32) / NX); }

// ------------------------------------------------------------------------------------------ registration
__device__ __forceinline__ uint32_t hw_xcc_id() {
  uint32_t v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 15u;
}

// Every workgroup publishes (epoch, hardware XCD id); wave 0 of each then reads all G words and derives
// the XCD rank X (rank of its id among the ids present), its slot s (workgroups of the same id with a
// smaller index), n (workgroups of its XCD), NX and n0 (workgroups of rank 0).  G <= 512.
__device__ __forceinline__ bool xcd_register(const TickArgs& a, TickLds& L) {
  constexpr int EPL = 8;
  const int G = gridDim.x;
  if (tix() == 0) st_dev(a.reg + blockIdx.x, (a.epoch << 8) | (uint64_t)hw_xcc_id());
  if (tix() < WAVE) {
    const int lane = tix();
    uint32_t xc[EPL];
    bool have[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      have[e] = e * WAVE + lane >= G;
      xc[e] = 0xffu;
    }
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    bool ok = true;
    for (uint32_t spin = 0;; ++spin) {
      bool all = true;
      // all of the lane's words loaded, unconditionally, before any is checked (a lane past the grid loads word 0
      // and ignores it)
      uint64_t v[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) v[e] = ld_dev(a.reg + (e * WAVE + lane < G ? e * WAVE + lane : 0));
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        if (!have[e]) {
          if ((v[e] >> 8) == a.epoch) {
            have[e] = true;
            xc[e] = (uint32_t)(v[e] & 0xffu);
          } else {
            all = false;
          }
        }
      }
      if (__all(all)) break;
      __builtin_amdgcn_s_sleep(1);
      if (timed_out(a, t0, spin)) {
        if (lane == 0) st_dev(a.status, fail_tag(a));
        ok = false;
        break;
      }
    }
    if (ok) {
      const int w = blockIdx.x;
      uint32_t sel = 0;
#pragma unroll
      for (int e = 0; e < EPL; ++e)
        if (e == w / WAVE) sel = xc[e];
      const uint32_t mine = (uint32_t)__builtin_amdgcn_readlane((int)sel, w % WAVE);
      int X = 0, NX = 0, n = 0, s = 0, n0 = 0;
      for (uint32_t x = 0; x < 16; ++x) {
        int cnt = 0;
#pragma unroll
        for (int e = 0; e < EPL; ++e) cnt += __popcll(__ballot(xc[e] == x));
        if (cnt > 0) {
          if (NX == 0) n0 = cnt;
          if (x < mine) ++X;
          ++NX;
        }
        if (x == mine) n = cnt;
      }
#pragma unroll
      for (int e = 0; e < EPL; ++e) s += __popcll(__ballot(xc[e] == mine && e * WAVE + lane < w));
      if (lane == 0) {
        L.X = X;
        L.s = s;
        L.n = n;
        L.NX = NX;
        L.n0 = n0;
        if (NX > NXR) ok = false;
      }
    }
    if (lane == 0) L.ok = ok;
  }
  __syncthreads();
  const bool ok = L.ok;
  __syncthreads();
  return ok;
}

// ------------------------------------------------------------------------------------------ staging
// Stage rows [m0, m0+rows) x K columns (K/8 <= 64 chunks of 16 bytes) of a row-major bf16 activation [M][ld]
// produced in this launch into L.x with direct global->LDS loads (device scope; one instruction per row: lane l
// brings columns 8l..8l+7, so an instruction reads whole 128-byte lines), columns K..511 set to zero, and, when
// ssq is given, the RMSNorm row scales r[row] = 1/sqrt(mean(h^2) + eps) from the per-16-column sums of squares
// ssq[tile][Ms] into L.r.  extra() issues the caller's own direct loads after the sums of squares (a register load
// issued after direct loads made the compiler wait for those first).  Every load is issued before any is waited
// for; ends with a barrier.  Rows past `rows` are left as they are: an MFMA output row depends only on its input
// row, and those rows are never stored.
struct NoLoads {
  __device__ void operator()() const {}
};
template <typename Extra = NoLoads>
__device__ __forceinline__ void stage(const uint16_t* src, int ld, int m0, int rows, int K, const float* ssq, int Ms,
                                      int Kn, float eps, TickLds& L, Extra extra = Extra()) {
  const int tid = tix(), wave = tid >> 6, lane = tid & 63;
  const int cpr = K / 8;  // chunks per row
  // the sums of squares first: loads complete in issue order, so these arrive while the rows are in flight
  const int g = tid & 15, rw = tid >> 4, ntn = Kn / 16;  // ntn <= 32
  float s0[MTMAX], s1[MTMAX];
  if (ssq) {
#pragma unroll
    for (int p = 0; p < MTMAX; ++p) {
      const int i = rw + 16 * p;
      s0[p] = i < rows && g < ntn ? ld_dev_f(ssq + (int64_t)g * Ms + m0 + i) : 0.f;
      s1[p] = i < rows && g + 16 < ntn ? ld_dev_f(ssq + (int64_t)(g + 16) * Ms + m0 + i) : 0.f;
    }
  }
  extra();  // the caller's own direct loads
  if (lane < cpr) {
    const uint16_t* row0 = src + (int64_t)m0 * ld + lane * 8;
    for (int m = wave; m < rows; m += 4) load_lds16<true>(row0 + (int64_t)m * ld, &L.u.p.x[m][0]);
  } else {
    for (int m = wave; m < rows; m += 4) *reinterpret_cast<uint4*>(&L.u.p.x[m][lane * 8]) = make_uint4(0, 0, 0, 0);
  }
  vm_wait_all();  // every load above (and any weight loads issued earlier) is complete
  if (ssq) {
#pragma unroll
    for (int p = 0; p < MTMAX; ++p) {
      const float sum = row_sum16(s0[p] + s1[p]);
      const int i = rw + 16 * p;
      if (g == 0) L.r[i] = i < rows ? 1.0f / sqrtf(sum / (float)Kn + eps) : 0.f;
    }
  }
  __syncthreads();
}

// ------------------------------------------------------------------------------------------ projections
// LDS operand reads of a projection row tile: every read is issued before one wait.  Written as one asm block
// (which waits for its own reads) because the compiler, short of registers in this kernel, otherwise reuses one
// register quad for all of them and waits after each read, which serialises their latencies.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// x[i] = 16 bytes at p + 64 i, i < 16
__device__ __forceinline__ void lds_read_16x64(const void* p, u32x4_t (&x)[16]) {
  asm volatile(
      "ds_read_b128 %0, %16 offset:0\n\t"
      "ds_read_b128 %1, %16 offset:64\n\t"
      "ds_read_b128 %2, %16 offset:128\n\t"
      "ds_read_b128 %3, %16 offset:192\n\t"
      "ds_read_b128 %4, %16 offset:256\n\t"
      "ds_read_b128 %5, %16 offset:320\n\t"
      "ds_read_b128 %6, %16 offset:384\n\t"
      "ds_read_b128 %7, %16 offset:448\n\t"
      "ds_read_b128 %8, %16 offset:512\n\t"
      "ds_read_b128 %9, %16 offset:576\n\t"
      "ds_read_b128 %10, %16 offset:640\n\t"
      "ds_read_b128 %11, %16 offset:704\n\t"
      "ds_read_b128 %12, %16 offset:768\n\t"
      "ds_read_b128 %13, %16 offset:832\n\t"
      "ds_read_b128 %14, %16 offset:896\n\t"
      "ds_read_b128 %15, %16 offset:960\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3]), "=&v"(x[4]), "=&v"(x[5]), "=&v"(x[6]), "=&v"(x[7]), "=&v"(x[8]), "=&v"(x[9]), "=&v"(x[10]), "=&v"(x[11]), "=&v"(x[12]), "=&v"(x[13]), "=&v"(x[14]), "=&v"(x[15])
      : "v"(lds_addr(p))
      : "memory");
}
// x[j] = 16 bytes at p + 256 j, j < 4
__device__ __forceinline__ void lds_read_4x256(const void* p, u32x4_t (&x)[4]) {
  asm volatile(
      "ds_read_b128 %0, %4 offset:0\n\t"
      "ds_read_b128 %1, %4 offset:256\n\t"
      "ds_read_b128 %2, %4 offset:512\n\t"
      "ds_read_b128 %3, %4 offset:768\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3])
      : "v"(lds_addr(p))
      : "memory");
}
__device__ __forceinline__ uint4 as_u4(u32x4_t v) { return make_uint4(v.x, v.y, v.z, v.w); }

// A projection unit is one 16-column tile over a range of nkb <= 16 k-blocks; wave w owns the unit's
// k-blocks i = w, w+4, w+8, w+12, whose 1 KiB weight blocks it holds in registers.
__device__ __forceinline__ void load_unit_w(const uint4* __restrict__ wtile, int kb0, int nkb, uint4 w[4]) {
  const int wave = tix() >> 6, lane = tix() & 63;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = wave + 4 * j;
    w[j] = i < nkb ? ld_global(wtile + (int64_t)(kb0 + i) * WAVE + lane) : make_uint4(0, 0, 0, 0);
  }
}

// acc = staged x (mt_n row tiles, k-blocks 0..nkb-1 of the unit's range) times the unit's weights, summed over
// the 4 waves through LDS and handed to epi(mt, C-layout values, c, grp) by wave mt % 4.  The row tiles are a
// run-time loop (one copy of the code and of the epilogue, which keeps the kernel small enough for the
// instruction cache); inside a row tile every LDS operand is read before the MFMAs.  The k-blocks past nkb
// multiply zero weights by the zero columns stage() leaves there, so the loop has no branches (a branch per
// k-block makes the compiler wait for each LDS read before issuing the next).
template <typename Epi>
__device__ __forceinline__ void unit_gemm(const uint4 w[4], int nkb, int mt_n, TickLds& L, Epi epi) {
  const int wave = tix() >> 6, lane = tix() & 63;
  const int c = lane & 15, grp = lane >> 4;
  const bool any = nkb > 0;  // nothing staged otherwise
#pragma unroll 1
  for (int mt = 0; mt < mt_n; ++mt) {
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    if (any) {
      u32x4_t xa[4];
      lds_read_4x256(&L.u.p.x[mt * 16 + c][wave * 32 + 8 * grp], xa);
#pragma unroll
      for (int j = 0; j < 4; ++j) acc = mfma_bf16(as_u4(xa[j]), w[j], acc);
    }
    L.u.p.red[wave][mt][lane] = acc;
  }
  __syncthreads();
#pragma unroll 1
  for (int mt = wave; mt < mt_n; mt += 4) {
    const f32x4 s = L.u.p.red[0][mt][lane] + L.u.p.red[1][mt][lane] + L.u.p.red[2][mt][lane] + L.u.p.red[3][mt][lane];
    epi(mt, s, c, grp);
  }
  __syncthreads();
}

// The row-split projections (O, F1, D) load the weights of IPF items of a workgroup (items it0 + j n) together, so
// that with several row blocks the second item's weights are not fetched after the first item's product.
constexpr int IPF = 2;
__device__ __forceinline__ void pick_w(const uint4 (&w)[IPF][4], int j, uint4 (&out)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = w[0][i];
#pragma unroll
  for (int jj = 1; jj < IPF; ++jj)
    if (j == jj)
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = w[jj][i];
}

// One wave per projection unit: the wave holds the unit's 16-column tile for every k-block (K <= 512) in
// registers and multiplies all staged row tiles.
__device__ __forceinline__ void load_unit_w_full(const uint4* __restrict__ wtile, int nkb, uint4 w[16]) {
  const int lane = tix() & 63;
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i] = i < nkb ? ld_global(wtile + (int64_t)i * WAVE + lane) : make_uint4(0, 0, 0, 0);
}

// Per row tile (a run-time loop): the 16 LDS operands are read first, then the MFMAs run on two accumulators
// (even and odd k-blocks) so that consecutive MFMAs do not depend on each other.  As in unit_gemm, k-blocks past
// the staged width multiply zeros, without branches.
template <typename Epi>
__device__ __forceinline__ void wave_gemm(const uint4 w[16], int mt_n, TickLds& L, Epi epi) {
  const int lane = tix() & 63, c = lane & 15, grp = lane >> 4;
#pragma unroll 1
  for (int mt = 0; mt < mt_n; ++mt) {
    u32x4_t xa[16];
    lds_read_16x64(&L.u.p.x[mt * 16 + c][8 * grp], xa);
    f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
#pragma unroll
    for (int i = 0; i < 16; i += 2) {
      acc0 = mfma_bf16(as_u4(xa[i]), w[i], acc0);
      acc1 = mfma_bf16(as_u4(xa[i + 1]), w[i + 1], acc1);
    }
    epi(mt, acc0 + acc1, c, grp);
  }
}

// ------------------------------------------------------------------------------------------ reductions
// Pieces of the cross-XCD reductions: column tile i (16 columns) of the residual belongs to the XCD of rank X
// with tile_lo(X) <= i < tile_lo(X + 1); its rows are cut into tp.rblk blocks, rows [piece_row(rb),
// piece_row(rb + 1)).  Piece (i, rb) is the q-th of its XCD, q = (i - tile_lo(X)) * rblk + rb, and goes to the
// workgroup of slot q mod n, in the embedding and in every reduction, so each residual element is always
// updated by the same workgroup.  Its flag is f[(i * rblk + rb) * FPAD].
__device__ __forceinline__ int tile_lo(int X, int NX, int nt) { return X * nt / NX; }
__device__ __forceinline__ int piece_row(const TickParams& tp, int rb) { return rb * tp.M / tp.rblk; }

// Piece (i, rb): h[m][i] += sum over XCDs x (fixed order) of part[x][i][m][:] for its rows m, where part holds
// stamped words.  Thread t owns the elements e = e_lo + t + 256 k (e = m*16 + c, k < EB); all of its words are
// loaded before any is checked, then it polls its own stale words until their stamps are right.  The new values
// go to the residual hres, to the row-major bf16 copy xb and the per-row sums of squares ssq (device-scope
// stores: every XCD reads them), and, if given, to hidden; then the piece's flag is published.
constexpr int EB = 5;  // element batches per pass: 80 rows in one pass
__device__ __forceinline__ bool reduce_piece(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, int i,
                                             int rb, const uint64_t* part, uint16_t* xb, float* ssq, uint64_t* flag,
                                             float* hidden_l, TickLds& L) {
  const int NX = uni(L.NX), nt = dm.d / 16;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const uint32_t st32 = (uint32_t)st;
  float* hres = a.hres + (int64_t)i * tp.Mp * 16;
  const int64_t xs = (int64_t)nt * tp.Mp * 16;  // words between the partials of two XCDs
  const int e_lo = piece_row(tp, rb) * 16, e_hi = piece_row(tp, rb + 1) * 16;
  bool ok = true;
  for (int e0 = e_lo; e0 < e_hi && ok; e0 += EB * NTHR) {
    // Batch k is skipped as a whole when none of its elements exists; in a partial batch the threads past the
    // end load the last element (in bounds) and ignore it, so no load depends on a per-thread branch.  Words
    // are used only where use[k] bit x is set (x < NX and the element exists).
    uint64_t v[EB][NXR];
    float hold[EB];
    uint32_t use[EB], pend[EB];
#pragma unroll
    for (int k = 0; k < EB; ++k) {
      const int e = e0 + k * NTHR + tix();
      const uint64_t* src = part + (int64_t)i * tp.Mp * 16 + min(e, e_hi - 1);
      use[k] = e < e_hi ? (1u << NX) - 1 : 0u;
      if (e0 + k * NTHR < e_hi) {
#pragma unroll
        for (int x = 0; x < NXR; ++x) v[k][x] = ld_dev(src + (x < NX ? x : 0) * xs);
        hold[k] = ld_dev_f(hres + min(e, e_hi - 1));
      } else {
#pragma unroll
        for (int x = 0; x < NXR; ++x) v[k][x] = 0;
        hold[k] = 0.f;
      }
    }
    bool pending = false;
#pragma unroll
    for (int k = 0; k < EB; ++k) {
      pend[k] = 0;
#pragma unroll
      for (int x = 0; x < NXR; ++x)
        if ((uint32_t)(v[k][x] >> 32) != st32) pend[k] |= 1u << x;
      pend[k] &= use[k];
      pending = pending || pend[k] != 0;
    }
    if (pending) {
      const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
      for (uint32_t spin = 0; pending; ++spin) {
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int k = 0; k < EB; ++k) {
          const uint64_t* src = part + (int64_t)i * tp.Mp * 16 + e0 + k * NTHR + tix();
#pragma unroll
          for (int x = 0; x < NXR; ++x)
            if (pend[k] & (1u << x)) v[k][x] = ld_dev(src + x * xs);
        }
        pending = false;
#pragma unroll
        for (int k = 0; k < EB; ++k) {
#pragma unroll
          for (int x = 0; x < NXR; ++x)
            if ((uint32_t)(v[k][x] >> 32) == st32) pend[k] &= ~(1u << x);
          pending = pending || pend[k] != 0;
        }
        if (pending && timed_out(a, t0, spin)) {
          st_dev(a.status, fail_tag(a));
          ok = false;
          break;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < EB; ++k) {
      const int e = e0 + k * NTHR + tix();
      const bool in = use[k] != 0;
      const int m = e >> 4, c = e & 15;
      float acc = 0.f;
#pragma unroll
      for (int x = 0; x < NXR; ++x)
        if (use[k] & (1u << x)) acc += __uint_as_float((uint32_t)v[k][x]);
      const float hv = hold[k] + acc;
      if (in) {
        st_dev_f(hres + e, hv);
        if (hidden_l) hidden_l[(int64_t)m * dm.d + i * 16 + c] = hv;
      }
      const float vn = xor1(hv);
      if (in && (c & 1) == 0)
        st_dev(reinterpret_cast<uint32_t*>(xb + (int64_t)m * dm.d + i * 16 + c), pack_bf16x2(hv, vn));
      const float sq = row_sum16(hv * hv);
      if (in && c == 0) st_dev_f(ssq + (int64_t)i * tp.Ms + m, sq);
    }
  }
  stores_done();
  __syncthreads();
  if (tix() == 0) st_dev(flag + ((int64_t)i * tp.rblk + rb) * FPAD, st);
  return __syncthreads_and(ok);
}

// ------------------------------------------------------------------------------------------ embed
// The owner of each residual piece copies the tokens' values into the residual, its bf16 copy and sums of squares
// (the input of layer 0) and publishes the piece; rotary rows m = s, s + n, ... (fp64 angles) are written in every
// XCD for its own use.
__device__ __forceinline__ void phase_embed(const TickArgs& a, const TickParams& tp, const Dims& dm, TickLds& L) {
  const int X = uni(L.X), s = uni(L.s), n = uni(L.n), NX = uni(L.NX), d = dm.d, M = tp.M, half = dm.Dh / 2;
  const int nt = d / 16, t0 = tile_lo(X, NX, nt), t1 = tile_lo(X + 1, NX, nt);
  const uint64_t st = stamp_of(a, -1, dm.n_layers);
  float* hres = a.hres;
  uint16_t* xb = a.xb_out;
  float* ssq = a.ssq_out;
  float* rope = a.rope + (int64_t)X * a.x_stride_r;
  for (int q = s; q < (t1 - t0) * tp.rblk; q += n) {
    const int i = t0 + q / tp.rblk, rb = q % tp.rblk;
    // whole rows of 16 elements per 16-lane group, so the neighbour and row-sum shuffles stay inside live lanes
    for (int e = piece_row(tp, rb) * 16 + tix(); e < piece_row(tp, rb + 1) * 16; e += NTHR) {
      const int m = e >> 4, c = e & 15;
      const int64_t idx = (int64_t)m * d + i * 16 + c;
      const float v = a.tok_dtype == FSX_BF16 ? bf16_to_f32(((const uint16_t*)a.tokens)[idx]) : ((const float*)a.tokens)[idx];
      st_dev_f(hres + (int64_t)i * tp.Mp * 16 + e, v);
      const float vn = xor1(v);
      if ((c & 1) == 0) st_dev(reinterpret_cast<uint32_t*>(xb + (int64_t)m * d + i * 16 + c), pack_bf16x2(v, vn));
      const float sq = row_sum16(v * v);
      if (c == 0) st_dev_f(ssq + (int64_t)i * tp.Ms + m, sq);
    }
    stores_done();
    __syncthreads();
    if (tix() == 0) st_dev(a.f_out + ((int64_t)i * tp.rblk + rb) * FPAD, st);
  }
  for (int m = s; m < M; m += n) {
    const int b = m / tp.S, t = m % tp.S;
    for (int j = tix(); j < half; j += NTHR) {
      double cs = 1.0, sn = 0.0;
      if (dm.rope_base > 0.f) {
        const double ang = (double)(tp.pos[b] + t) * pow((double)dm.rope_base, -2.0 * (double)j / (double)dm.Dh);
        cs = cos(ang);
        sn = sin(ang);
      }
      st_loc_f(rope + ((int64_t)m * half + j) * 2, (float)cs);
      st_loc_f(rope + ((int64_t)m * half + j) * 2 + 1, (float)sn);
    }
  }
  stores_done();
  __syncthreads();
  if (tix() == 0) st_loc(a.f_rope + ((int64_t)X * XFLAGS + s) * FPAD, st);
}

// ------------------------------------------------------------------------------------------ Q
// Units of XCD X: u = (local head hl, section sec (q, k, v), 16-column tile t), 24 per head of width 128.
// Workgroup s takes units s, s + n, ...; its k-th unit goes to wave k % 4, which holds the unit's weights in
// registers (loaded before the wait).  Each unit publishes a flag once its columns are written.  When each
// attention segment has a workgroup of its own (plan mode 1) and the other workgroups have a wave for every unit,
// those take all units, so that the attention workgroups start streaming their cache tiles at once.
__device__ __forceinline__ bool phase_qkv(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  const int X = uni(L.X), s = uni(L.s), n = uni(L.n), NX = uni(L.NX);
  const int d = dm.d, M = tp.M, A = dm.A, H = dm.H, half = DH / 2, nt = d / 16, R = row_blocks(M);
  const int wave = uni(tix() >> 6);  // scalar, so the unit's section is a uniform branch
  const int h0 = head_lo(X, NX, H), nh = head_lo(X + 1, NX, H) - h0;
  const int n_units = 24 * nh;
  const LayerW W = layer_w(a, dm, l);
  const int KB = d / 32;
  const float qs = LOG2E / sqrtf((float)DH);
  const uint16_t* xb = a.xb_out;
  const float* ssq = a.ssq_out;
  const float* rope = a.rope + (int64_t)X * a.x_stride_r;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const int nseg = tp.B * nh, nq = n - nseg;  // attention workgroups, and the others
  const bool spare = uni(L.amode) == 1 && nq > 0 && n_units <= 4 * nq;
  const int s0 = spare ? s - nseg : s, nw = spare ? nq : n;  // this workgroup's index among the Q workgroups
  // With several row blocks (and n a multiple of R) workgroup s takes row block s mod R only, staged once, and the
  // units s / R + (n / R)(w + 4k); otherwise every row block of units s0 + nw (w + 4k).
  const bool by_rows = R > 1 && !spare && n % R == 0;
  const int rb0 = by_rows ? s % R : 0, rb1 = by_rows ? rb0 + 1 : R;
  const int ub = by_rows ? s / R : s0, us = by_rows ? n / R : nw;
  bool waited = false;
  int staged = -1;  // row block in L.x
  uint4 w[16], wn[16];
  {
    const int u = ub + us * wave;
    if (s0 >= 0 && u < n_units) {
      const int tile = ((u % 24) / 8) * (A / 16) + (h0 + u / 24) * (DH / 16) + u % 8;
      load_unit_w_full(W.wqkv + (int64_t)tile * KB * WAVE, KB, w);
    }
  }
  for (int u0 = ub; s0 >= 0 && u0 < n_units; u0 += 4 * us) {
    const int u = u0 + wave * us;  // this wave's unit in this round
    const bool mine = u < n_units;
    const int hl = u / 24, sec = (u % 24) / 8, t = u % 8;
    const int h = h0 + hl;
    const int tile = sec * (A / 16) + h * (DH / 16) + t;  // 16-row tile of packed [q; k; v]
    // the next round's weights stream in during this round (one row block: the rows are staged once)
    const int un = u + 4 * us;
    if (by_rows && un < n_units) {
      const int tn = ((un % 24) / 8) * (A / 16) + (h0 + un / 24) * (DH / 16) + un % 8;
      load_unit_w_full(W.wqkv + (int64_t)tn * KB * WAVE, KB, wn);
    }
    if (!waited) {
      TICK_SUB(l, 0);
      bool ok = wg_wait(a.f_out, nt * tp.rblk, stamp_of(a, l - 1, dm.n_layers), a, L);
      if (ok && l == 0) ok = wg_wait(a.f_rope + (int64_t)X * XFLAGS * FPAD, n, stamp_of(a, -1, dm.n_layers), a, L);
      if (!ok) return false;
      waited = true;
      TICK_SUB(l, 1);
    }
    const int nl0 = h * DH + t * 16;  // first column of the unit inside its section
    for (int r = rb0; r < rb1; ++r) {
      const int m0 = r * MTMAX * 16, rows = min(MTMAX * 16, M - m0), mt_n = (rows + 15) / 16;
      // this wave's rotary slice: rope[row][8t .. 8t+7][2] (64 bytes per row), 16 rows per direct load
      auto rope_loads = [&]() {
        if (mine && sec < 2) {
          const int ln = tix() & 63;
          for (int r0 = 0; r0 < rows; r0 += 16) {
            const int row = min(m0 + r0 + (ln >> 2), M - 1);
            load_lds16<true>(rope + ((int64_t)row * half + 8 * t) * 2 + (ln & 3) * 4, &L.u.p.rq[wave][r0][0][0]);
          }
        }
      };
      if (staged != r) {
        stage(xb, d, m0, rows, d, ssq, tp.Ms, d, dm.eps, L, rope_loads);
        staged = r;
      } else {
        rope_loads();  // the wave's own slice only; read once its loads have landed
        vm_wait_all();
      }
      TICK_SUB(l, 2);
      if (mine) {
        wave_gemm(w, mt_n, L, [&](int mt, f32x4 sacc, int c, int grp) {
          // element i of the C tile is row rb + i of the chunk, column nl0 + c
          const int rb = mt * 16 + 4 * grp, nl = nl0 + c;
          const f32x4 rs = *reinterpret_cast<const f32x4*>(&L.r[rb]);  // RMSNorm row scales
          if (sec == 2) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float v = sacc[i] * rs[i];
              const float other = xor1(v);
              if ((c & 1) == 0 && m0 + rb + i < M)
                st_loc(reinterpret_cast<uint32_t*>(a.vself + (int64_t)(m0 + rb + i) * A + nl), pack_bf16x2(v, other));
            }
          } else {
            float2 cs[4];  // (cos, sin) of the pair in this lane's column, per row
#pragma unroll
            for (int i = 0; i < 4; ++i) cs[i] = *reinterpret_cast<const float2*>(&L.u.p.rq[wave][rb + i][c & 7][0]);
            const int p = nl % DH;
            const int j = 8 * (p / 16) + (c & 7);
            const int dch = c < 8 ? j : half + j;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float v = sacc[i] * rs[i];
              const float partner = xor8(v);
              const float rr = c < 8 ? v * cs[i].x - partner * cs[i].y : v * cs[i].x + partner * cs[i].y;
              const int row = m0 + rb + i;
              const int64_t o = (int64_t)row * A + h * DH + dch;
              if (sec == 0) {
                if (row < M) st_loc_f(a.q + o, rr * qs);
              } else {
                const float nb = xor1(rr);  // neighbouring channel dch+1 sits in lane c+1
                if ((c & 1) == 0 && row < M) st_loc(reinterpret_cast<uint32_t*>(a.kself + o), pack_bf16x2(rr, nb));
              }
            }
          }
        });
      }
      if (!by_rows) __syncthreads();  // the next chunk overwrites the staged rows
    }
    // publish this wave's unit: flag (tile, r) for each of its row blocks
    stores_done();
    if (mine && (tix() & 63) == 0)
      for (int r = rb0; r < rb1; ++r) st_loc(a.f_q + ((int64_t)tile * R + r) * FPAD, st);
    if (by_rows) {
#pragma unroll
      for (int i = 0; i < 16; ++i) w[i] = wn[i];
    } else if (u0 + 4 * us < n_units) {
      const int un2 = u + 4 * us;
      if (un2 < n_units) {
        const int tn = ((un2 % 24) / 8) * (A / 16) + (h0 + un2 / 24) * (DH / 16) + un2 % 8;
        load_unit_w_full(W.wqkv + (int64_t)tn * KB * WAVE, KB, w);
      }
    }
  }
  if (by_rows) __syncthreads();  // the next phase overwrites the staged rows
  TICK_SUB(l, 3);
  return true;
}

// ------------------------------------------------------------------------------------------ A
// Registers of one 32-row tile, as read from its LDS slots; the kind says how (0: bf16 rows, 1: fp8 rows).  bf16: k[rt*4 + kb] = K row r0+16rt+c, channels 32kb+8grp..+7; fp8: k[rt*2 + h] = K row
// r0+16rt+c, channels 64h+16grp..+15 (16 bytes; the k-blocks of the score MFMA then hold channels 64(kb/2) + 16grp +
// 8(kb%2) + j, and the fp16 queries use the same order).  Kinds 0, 1: v[j] = V row r0 + (j<4 ? 4grp+j : 16+4grp+j-4),
// channels 8c..8c+7 (fp8 tiles hold the codes, decoded when the tile is used); the P V output then holds channel
// 8c + k in accumulator k.  (The V operand is transposed in registers: LDS transposed reads, ds_read_b64_tr_b16,
// gave run-to-run differences in the results of the workgroup-shared ring below, so the kernel does not use them.)
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

// Own-row tile (the expert's rows [r0, r0+32) of S, bf16, produced in this launch): device-scope loads.
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

// Query fragments of query tiles tts[j] (j < nq) of agent b, head h (16 queries x 128 channels each, B operand
// of S^T = K Q^T): bf16 in plain channel order (F16 = false), or fp16 in the channel order of fp8 key tiles.
template <int NQ, bool F16>
__device__ __forceinline__ void load_q(const TickArgs& a, const TickParams& tp, const Dims& dm, int b, int h,
                                       const int (&tts)[NQ], int nq, uint4 (&q)[NQ][4]) {
  const int lane = tix() & 63, grp = lane >> 4;
#pragma unroll
  for (int tt = 0; tt < NQ; ++tt) {
    const int t = tts[tt] * 16 + (lane & 15);
    const bool tv = tt < nq && t < tp.S;
    const float* row = a.q + ((int64_t)b * tp.S + (tv ? t : 0)) * dm.A + (int64_t)h * DH;
    // every load first, then the conversions
    float4 lo[4], hi[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int ch = F16 ? 64 * (kb >> 1) + 16 * grp + 8 * (kb & 1) : 32 * kb + 8 * grp;
      lo[kb] = ld_dev_f4(row + ch);
      hi[kb] = ld_dev_f4(row + ch + 4);
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if (!tv) lo[kb] = hi[kb] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (F16)
        q[tt][kb] = make_uint4(pack_f16x2(lo[kb].x, lo[kb].y), pack_f16x2(lo[kb].z, lo[kb].w),
                               pack_f16x2(hi[kb].x, hi[kb].y), pack_f16x2(hi[kb].z, hi[kb].w));
      else
        q[tt][kb] = make_uint4(pack_bf16x2(lo[kb].x, lo[kb].y), pack_bf16x2(lo[kb].z, lo[kb].w),
                               pack_bf16x2(hi[kb].x, hi[kb].y), pack_bf16x2(hi[kb].z, hi[kb].w));
    }
  }
}

// 2^x by the hardware instruction (about 1 ulp; results below the normal range are flushed to zero, which only
// drops probabilities under 2^-126).
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// MFMA operands of one raw tile: K fragments kf (A operand of S^T = K Q^T) and V transposed to per-channel
// vectors vt (B operand of O += P V); fp8 codes are decoded to fp16 (exact).
template <int KT>
__device__ __forceinline__ void tile_operands(const RawTile<KT>& t, uint4 (&kf)[8], uint4 (&vt)[8]) {
  uint4 vr[8];
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
  transpose8x8_b16(vr, vt);
}

// Online-softmax update of NJ query-tile states ("jobs") with one tile whose rows r0.. (valid below i1) are in t;
// job j takes part when bit j of ACT is set, and qf(j, kb) returns the B-operand fragment kb of its queries.  The
// steps run for all jobs together (scores, then maxima, then one rescale test, then probabilities, then P V), so
// the independent work of the jobs can overlap.  fp8 tiles (KT 1) are decoded to fp16 (exact) and use fp16 MFMA;
// their key scale multiplies the fp32 scores (the value scale is applied to the output once, after the cache
// tiles).  The running max of a query only moves when a score exceeds it by more than 2^8 (log2 units), so the
// accumulators are rescaled rarely; probabilities stay below 2^8.  Rows at or past i1 are masked only in a tile
// that reaches past i1.
constexpr float RESCALE_LOG2 = 8.0f;
template <int KT, int NJ, int ACT, typename QF>
__device__ __forceinline__ void tile_jobs(const RawTile<KT>& t, QF qf, int r0, int i1, float kscale,
                                          f32x4 (&o)[NJ][8], float (&m_run)[NJ], float (&l_run)[NJ]) {
  constexpr bool F16 = KT == 1;
  const int lane = tix() & 63, grp = lane >> 4;
  uint4 kf[8], vt[8];
  tile_operands<KT>(t, kf, vt);
  f32x4 s[NJ][2];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) s[j][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (ACT >> j & 1) {
        const uint4 qk = qf(j, k);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          s[j][rt] = F16 ? mfma_f16(kf[rt * 4 + k], qk, s[j][rt]) : mfma_bf16(kf[rt * 4 + k], qk, s[j][rt]);
      }
  if (KT == 1)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) s[j][rt] *= kscale;
  if (r0 + 32 > i1) {
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (r0 + 16 * rt + 4 * grp + i >= i1) s[j][rt][i] = -INFINITY;
  }
  float mx[NJ];
  bool grow = false;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    mx[j] = -INFINITY;
    if (ACT >> j & 1) {
      mx[j] = vmax3(vmax3(s[j][0][0], s[j][0][1], s[j][0][2]), vmax3(s[j][0][3], s[j][1][0], s[j][1][1]),
                    vmax(s[j][1][2], s[j][1][3]));
      mx[j] = rows_max(mx[j]);
      grow = grow || mx[j] > m_run[j] + RESCALE_LOG2;
    }
  }
  if (__any(grow)) {
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (ACT >> j & 1) {
        const float m_new = mx[j] > m_run[j] + RESCALE_LOG2 ? mx[j] : m_run[j];
        const float alpha = exp2_fast(m_run[j] - m_new);
        l_run[j] *= alpha;
        m_run[j] = m_new;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float a_i = col_pick(alpha, grp, i);
#pragma unroll
          for (int k = 0; k < 8; ++k) o[j][k][i] *= a_i;
        }
      }
  }
  uint4 pf[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (ACT >> j & 1) {
      float p[8], ps = 0.f;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          p[rt * 4 + i] = exp2_fast(s[j][rt][i] - m_run[j]);
          ps += p[rt * 4 + i];
        }
      l_run[j] += ps;
      if (F16)
        pf[j] = make_uint4(pack_f16x2(p[0], p[1]), pack_f16x2(p[2], p[3]), pack_f16x2(p[4], p[5]),
                           pack_f16x2(p[6], p[7]));
      else
        pf[j] = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                           pack_bf16x2(p[6], p[7]));
    }
#pragma unroll
  for (int k = 0; k < 8; ++k)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (ACT >> j & 1) o[j][k] = F16 ? mfma_f16(pf[j], vt[k], o[j][k]) : mfma_bf16(pf[j], vt[k], o[j][k]);
}

// One query tile, two tiles at once (64 rows): the score MFMAs of both tiles are independent, one running-max
// update covers both, and both P V products accumulate into the same output.  Twice the data per dependent chain
// of the single-tile update (the wave is the only one on its SIMD, so nothing else hides that chain).  Tile a holds
// rows ra.. (valid below ia1), tile b rows rb.. (valid below ib1).
template <int KT>
__device__ __forceinline__ void tile_pair_compute(const RawTile<KT>& ta, const RawTile<KT>& tb, const uint4 (&q)[4],
                                                  int ra, int ia1, int rb, int ib1, float kscale, f32x4 (&o)[8],
                                                  float& m_run, float& l_run) {
  constexpr bool F16 = KT == 1;
  const int lane = tix() & 63, grp = lane >> 4;
  uint4 kfa[8], vta[8], kfb[8], vtb[8];
  tile_operands<KT>(ta, kfa, vta);
  tile_operands<KT>(tb, kfb, vtb);
  f32x4 s[4];  // rt 0, 1 of tile a; rt 0, 1 of tile b
#pragma unroll
  for (int j = 0; j < 4; ++j) s[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      s[rt] = F16 ? mfma_f16(kfa[rt * 4 + k], q[k], s[rt]) : mfma_bf16(kfa[rt * 4 + k], q[k], s[rt]);
      s[2 + rt] = F16 ? mfma_f16(kfb[rt * 4 + k], q[k], s[2 + rt]) : mfma_bf16(kfb[rt * 4 + k], q[k], s[2 + rt]);
    }
  }
  if (KT == 1)
#pragma unroll
    for (int j = 0; j < 4; ++j) s[j] *= kscale;
  if (ra + 32 > ia1 || rb + 32 > ib1) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if ((j < 2 ? ra : rb) + 16 * (j & 1) + 4 * grp + i >= (j < 2 ? ia1 : ib1)) s[j][i] = -INFINITY;
  }
  float mx = vmax3(vmax3(s[0][0], s[0][1], s[0][2]), vmax3(s[0][3], s[1][0], s[1][1]), vmax3(s[1][2], s[1][3], s[2][0]));
  mx = vmax3(mx, vmax3(s[2][1], s[2][2], s[2][3]), vmax3(s[3][0], s[3][1], vmax3(s[3][2], s[3][3], s[3][3])));
  mx = rows_max(mx);
  const bool grow = mx > m_run + RESCALE_LOG2;
  if (__any(grow)) {
    const float m_new = grow ? mx : m_run;
    const float alpha = exp2_fast(m_run - m_new);
    l_run *= alpha;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a_i = col_pick(alpha, grp, i);
#pragma unroll
      for (int k = 0; k < 8; ++k) o[k][i] *= a_i;
    }
  }
  float p[16], ps = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[j * 4 + i] = exp2_fast(s[j][i] - m_run);
      ps += p[j * 4 + i];
    }
  l_run += ps;
  uint4 pa, pb;
  if (F16) {
    pa = make_uint4(pack_f16x2(p[0], p[1]), pack_f16x2(p[2], p[3]), pack_f16x2(p[4], p[5]), pack_f16x2(p[6], p[7]));
    pb = make_uint4(pack_f16x2(p[8], p[9]), pack_f16x2(p[10], p[11]), pack_f16x2(p[12], p[13]), pack_f16x2(p[14], p[15]));
  } else {
    pa = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7]));
    pb = make_uint4(pack_bf16x2(p[8], p[9]), pack_bf16x2(p[10], p[11]), pack_bf16x2(p[12], p[13]),
                    pack_bf16x2(p[14], p[15]));
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    o[k] = F16 ? mfma_f16(pa, vta[k], o[k]) : mfma_bf16(pa, vta[k], o[k]);
    o[k] = F16 ? mfma_f16(pb, vtb[k], o[k]) : mfma_bf16(pb, vtb[k], o[k]);
  }
}

// write a wave's state (o in the PV C layout: accumulator k holds channel 8c + k of rows 4grp + i, m and the
// lane-partial l) to LDS slot w as [16 rows][128 channels] and (m, l)[16]
__device__ __forceinline__ void state_to_lds(float* stw, const f32x4 o[8], float m_run, float l_run) {
  const int lane = tix() & 63, c = lane & 15, grp = lane >> 4;
  const float lt = rows_sum(l_run);
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
  int b, h;
  bool final_out;   // the whole (agent, head): normalised output, else the partial state of slot `slot`
  int slot;
  int i0, i1;       // cache rows of this range
  int nct, nst;     // cache tiles, own-row tiles
  int rot;          // the unit's k-th cache tile in streaming order is tile (k + rot) mod nct of the range
  const char* kc;   // cache K/V base of (b, layer, head) (slot 0)
  const char* vc;
  int64_t rsb;      // bytes between two ring slots of the head
  const char* ks;   // own rows base of (b, head)
  const char* vs;
  float ksc, vsc;   // fp8 scales
};

// Where wave w's attention state goes: the start of its slots of the LDS tile ring.
static_assert(STW * 4 <= RSLOTS * RSLOT, "a wave's state fits in its ring slots");
__device__ __forceinline__ float* state_of(TickLds& L, int w) { return reinterpret_cast<float*>(&L.u.a.ring[w][0][0]); }
// Merge the 4 waves' LDS states of query tile tt: each thread owns (t, 8 channels).  If final, normalise into
// the attention output; else store the unnormalised partial of slot `item`.
__device__ __forceinline__ void merge_states(const TickArgs& a, const TickParams& tp, const Dims& dm,
                                             const AUnit& U, int tt, bool final_out, int64_t item, TickLds& L) {
  const int t = tix() >> 4, d0 = (tix() & 15) * 8;
  float Mx = -INFINITY;
#pragma unroll
  for (int w = 0; w < 4; ++w) Mx = fmaxf(Mx, state_of(L, w)[2048 + 2 * t]);
  float Ls = 0.f, acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float* stw = state_of(L, w);
    const float f = Mx == -INFINITY ? 0.f : exp2f(stw[2048 + 2 * t] - Mx);
    Ls += stw[2048 + 2 * t + 1] * f;
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += stw[t * 128 + d0 + k] * f;
  }
  if (final_out) {
    const int tok = tt * 16 + t;
    if (tok < tp.S) {
      const float inv = 1.0f / Ls;
      uint16_t* dst = a.attn + ((int64_t)U.b * tp.S + tok) * dm.A + (int64_t)U.h * DH + d0;
      st_loc16(dst, make_uint4(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                               pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)));
    }
  } else {
    float* po = a.att_o + (item * 16 + t) * 128 + d0;
    st_loc_f4(po, make_float4(acc[0], acc[1], acc[2], acc[3]));
    st_loc_f4(po + 4, make_float4(acc[4], acc[5], acc[6], acc[7]));
    if ((tix() & 15) == 0) {
      st_loc_f(a.att_ml + item * 32 + 2 * t, Mx);
      st_loc_f(a.att_ml + item * 32 + 2 * t + 1, Ls);
    }
  }
}

// Query tile tt of (agent b, head h): merge the partials of its nr ranges (fixed order) into the attention output;
// the partials are loaded 8 ranges at a time, every load issued before any is used.
__device__ __forceinline__ void combine_ranges(const TickArgs& a, const TickParams& tp, const Dims& dm, int b, int h,
                                               int slot0, int nr, int tt) {
  constexpr int RB = 8;
  const int t = tix() >> 4, d0 = (tix() & 15) * 8;
  const int H = dm.H;
  float Mx = -INFINITY, Ls = 0.f, acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.f;
  for (int r0 = 0; r0 < nr; r0 += RB) {
    float ms[RB], ls[RB];
    float4 v0[RB], v1[RB];
#pragma unroll
    for (int j = 0; j < RB; ++j) {
      ms[j] = -INFINITY;
      ls[j] = 0.f;
      v0[j] = v1[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (r0 + j < nr) {
        const int64_t item = (int64_t)(slot0 + r0 + j) * tp.n_tt + tt;
        ms[j] = ld_dev_f(a.att_ml + item * 32 + 2 * t);
        ls[j] = ld_dev_f(a.att_ml + item * 32 + 2 * t + 1);
        const float* po = a.att_o + (item * 16 + t) * 128 + d0;
        v0[j] = ld_dev_f4(po);
        v1[j] = ld_dev_f4(po + 4);
      }
    }
#pragma unroll
    for (int j = 0; j < RB; ++j) {
      if (r0 + j < nr) {
        const float mn = fmaxf(Mx, ms[j]);
        const float fa = Mx == -INFINITY ? 0.f : exp2f(Mx - mn), fb = ms[j] == -INFINITY ? 0.f : exp2f(ms[j] - mn);
        Ls = Ls * fa + ls[j] * fb;
        acc[0] = acc[0] * fa + v0[j].x * fb; acc[1] = acc[1] * fa + v0[j].y * fb;
        acc[2] = acc[2] * fa + v0[j].z * fb; acc[3] = acc[3] * fa + v0[j].w * fb;
        acc[4] = acc[4] * fa + v1[j].x * fb; acc[5] = acc[5] * fa + v1[j].y * fb;
        acc[6] = acc[6] * fa + v1[j].z * fb; acc[7] = acc[7] * fa + v1[j].w * fb;
        Mx = mn;
      }
    }
  }
  const int tok = tt * 16 + t;
  if (tok < tp.S) {
    const float inv = 1.0f / Ls;
    uint16_t* dst = a.attn + ((int64_t)b * tp.S + tok) * dm.A + (int64_t)h * DH + d0;
    st_loc16(dst, make_uint4(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                             pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)));
  }
}

// fp8 tile staged into LDS with direct loads (whole 128-byte rows: every instruction reads 8 full rows, which streams
// from HBM faster than the 64-byte row pieces of register loads in MFMA operand order).  Slot layout: K rows
// [32][128 B] then V rows [32][128 B]; the 16-byte chunk k of row r sits at chunk position k ^ ((r >> 1) & 7), so
// the 16 rows of a K fragment read fall in distinct banks.  Lane l of instruction q brings row 8q + l/8 into chunk
// position l % 8.  Rows past i1 repeat row i0 (masked in the update).
template <int NQI = 4>
__device__ __forceinline__ void stage_tile_fp8(const char* kb, const char* vb, int64_t rsb, int64_t start, int64_t cap,
                                               int i0, int r0, int i1, uint8_t* slot, int q0 = 0) {
  const int lane = tix() & 63, rl = lane >> 3, pc = lane & 7;
  asm volatile("" ::: "memory");  // after every read of the slot's previous tile
#pragma unroll
  for (int qq = 0; qq < NQI; ++qq) {
    const int q = q0 + qq, r = 8 * q + rl;
    int64_t row = start + (r0 + r < i1 ? r0 + r : i0);
    if (row >= cap) row -= cap;
    const int64_t off = row * rsb + 16 * (pc ^ ((r >> 1) & 7));
    load_lds16<false>(kb + off, slot + q * 1024);
    load_lds16<false>(vb + off, slot + 32 * DH + q * 1024);
  }
}
// The RawTile<1> fragments of a staged tile (see RawTile and stage_tile_fp8): K row 16rt + c, chunks 4h + grp; V
// rows 4grp + j (+16), bytes 8c..8c+7.  One asm block that waits for its own reads: reads the compiler sees after
// direct loads into the same LDS object make it wait for every pending direct load, the next tile's included.
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
// This lane's byte offsets (from the tile's first slot) of the reads of a staged tile, computed once per unit.
template <int KT>
struct TileLanes {
  // kind 0: K chunks k = 0..3, V rows j = 0..3; kind 1: K halves k = 0, 1, V rows j = 0..3
  uint32_t k[4], v[4];
};
template <int KT>
__device__ __forceinline__ TileLanes<KT> tile_lanes() {
  const int lane = tix() & 63, c = lane & 15, grp = lane >> 4;
  TileLanes<KT> tl;
  if constexpr (KT == 0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) tl.k[k] = c * 256 + 16 * ((4 * k + grp) ^ c);
#pragma unroll
    for (int j = 0; j < 4; ++j) tl.v[j] = 16 * 256 + (4 * grp + j) * 256 + 16 * (c ^ (4 * grp + j));
  } else {
    tl.k[0] = c * DH + 16 * (grp ^ (c >> 1));  // (r >> 1) & 7 == c >> 1 for r = 16 rt + c
    tl.k[1] = c * DH + 16 * ((4 + grp) ^ (c >> 1));
    tl.k[2] = tl.k[3] = 0;
    const uint32_t vb = 32 * DH + 4 * grp * DH + 8 * (c & 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) tl.v[j] = vb + j * DH + 16 * ((c >> 1) ^ (2 * grp + (j >> 1)));  // (r >> 1) & 7 == 2grp + j/2
  }
  return tl;
}
__device__ __forceinline__ void read_tile_fp8(const uint8_t* slot, const TileLanes<1>& tl, RawTile<1>& t) {
  const uint32_t s0 = lds_addr(slot);
  const uint32_t ak0 = s0 + tl.k[0], ak1 = s0 + tl.k[1];
  const uint32_t av0 = s0 + tl.v[0], av1 = s0 + tl.v[1], av2 = s0 + tl.v[2], av3 = s0 + tl.v[3];
  u32x4_t k0, k1, k2, k3;
  u32x2_t v0, v1, v2, v3, v4, v5, v6, v7;
  asm volatile(
      "ds_read_b128 %0, %12\n\t"
      "ds_read_b128 %1, %13\n\t"
      "ds_read_b128 %2, %12 offset:2048\n\t"
      "ds_read_b128 %3, %13 offset:2048\n\t"
      "ds_read_b64 %4, %14\n\t"
      "ds_read_b64 %5, %15\n\t"
      "ds_read_b64 %6, %16\n\t"
      "ds_read_b64 %7, %17\n\t"
      "ds_read_b64 %8, %14 offset:2048\n\t"
      "ds_read_b64 %9, %15 offset:2048\n\t"
      "ds_read_b64 %10, %16 offset:2048\n\t"
      "ds_read_b64 %11, %17 offset:2048\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k0), "=&v"(k1), "=&v"(k2), "=&v"(k3), "=&v"(v0), "=&v"(v1), "=&v"(v2), "=&v"(v3), "=&v"(v4), "=&v"(v5),
        "=&v"(v6), "=&v"(v7)
      : "v"(ak0), "v"(ak1), "v"(av0), "v"(av1), "v"(av2), "v"(av3)
      : "memory");
  t.k[0] = as_u4(k0);
  t.k[1] = as_u4(k1);
  t.k[2] = as_u4(k2);
  t.k[3] = as_u4(k3);
  const u32x2_t vv[8] = {v0, v1, v2, v3, v4, v5, v6, v7};
#pragma unroll
  for (int j = 0; j < 8; ++j) t.v[j] = make_uint2(vv[j].x, vv[j].y);
}

// bf16 tile staged into two LDS slots with direct loads of whole 256-byte rows (4 rows per instruction): slot h holds
// rows 16h .. 16h+15, K rows [16][256 B] then V rows [16][256 B]; the 16-byte chunk k of row r sits at chunk position
// k ^ (r & 15) (the 16 rows of a K fragment read, and the 4 rows of a V fragment read, fall in distinct banks).  Lane
// l of instruction q brings row 4q + l/16 into chunk position l % 16.  Rows past i1 repeat row i0.
template <int NQI = 8>
__device__ __forceinline__ void stage_tile_bf16(const char* kb, const char* vb, int64_t rsb, int64_t start, int64_t cap,
                                                int i0, int r0, int i1, uint8_t* slot, int q0 = 0) {
  const int lane = tix() & 63, rl = lane >> 4, pc = lane & 15;
  asm volatile("" ::: "memory");  // after every read of the slots' previous tile
#pragma unroll
  for (int qq = 0; qq < NQI; ++qq) {
    const int q = q0 + qq, r = 4 * q + rl;  // row of the tile, 0..31
    int64_t row = start + (r0 + r < i1 ? r0 + r : i0);
    if (row >= cap) row -= cap;
    const int64_t off = row * rsb + 16 * (pc ^ (r & 15));
    uint8_t* dst = slot + (q >> 2) * RSLOT + (q & 3) * 1024;
    load_lds16<false>(kb + off, dst);
    load_lds16<false>(vb + off, dst + 16 * DH * 2);
  }
}
// The RawTile<0> fragments of a staged bf16 tile: K row 16rt + c (slot rt, row c), channels 32k + 8grp (chunk 4k +
// grp); V rows 4grp + j (slot j / 4), channels 8c .. 8c+7 (chunk c).  One asm block that waits for its own reads.
__device__ __forceinline__ void read_tile_bf16(const uint8_t* slot, const TileLanes<0>& tl, RawTile<0>& t) {
  const uint32_t s0 = lds_addr(slot);
  uint32_t ak[4], av[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) ak[k] = s0 + tl.k[k];
#pragma unroll
  for (int j = 0; j < 4; ++j) av[j] = s0 + tl.v[j];
  u32x4_t k0, k1, k2, k3, k4, k5, k6, k7, v0, v1, v2, v3, v4, v5, v6, v7;
  asm volatile(
      "ds_read_b128 %0, %16\n\t"
      "ds_read_b128 %1, %17\n\t"
      "ds_read_b128 %2, %18\n\t"
      "ds_read_b128 %3, %19\n\t"
      "ds_read_b128 %4, %16 offset:8192\n\t"
      "ds_read_b128 %5, %17 offset:8192\n\t"
      "ds_read_b128 %6, %18 offset:8192\n\t"
      "ds_read_b128 %7, %19 offset:8192\n\t"
      "ds_read_b128 %8, %20\n\t"
      "ds_read_b128 %9, %21\n\t"
      "ds_read_b128 %10, %22\n\t"
      "ds_read_b128 %11, %23\n\t"
      "ds_read_b128 %12, %20 offset:8192\n\t"
      "ds_read_b128 %13, %21 offset:8192\n\t"
      "ds_read_b128 %14, %22 offset:8192\n\t"
      "ds_read_b128 %15, %23 offset:8192\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k0), "=&v"(k1), "=&v"(k2), "=&v"(k3), "=&v"(k4), "=&v"(k5), "=&v"(k6), "=&v"(k7), "=&v"(v0), "=&v"(v1),
        "=&v"(v2), "=&v"(v3), "=&v"(v4), "=&v"(v5), "=&v"(v6), "=&v"(v7)
      : "v"(ak[0]), "v"(ak[1]), "v"(ak[2]), "v"(ak[3]), "v"(av[0]), "v"(av[1]), "v"(av[2]), "v"(av[3])
      : "memory");
  const u32x4_t kk[8] = {k0, k1, k2, k3, k4, k5, k6, k7}, vv[8] = {v0, v1, v2, v3, v4, v5, v6, v7};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    t.k[i] = as_u4(kk[i]);
    t.v[i] = as_u4(vv[i]);
  }
}
template <int KT>
__device__ __forceinline__ void stage_tile(const char* kb, const char* vb, int64_t rsb, int64_t start, int64_t cap,
                                           int i0, int r0, int i1, uint8_t* slot) {
  if constexpr (KT == 0)
    stage_tile_bf16<8>(kb, vb, rsb, start, cap, i0, r0, i1, slot);
  else
    stage_tile_fp8<4>(kb, vb, rsb, start, cap, i0, r0, i1, slot);
}
// The expert's own rows [r0, r0+32) of (agent, head) (bf16, produced in this launch) staged in the bf16 tile layout
// by device-scope direct loads; instructions q0 .. q0+NQI-1 of the eight.  Rows at or past S repeat row 0.
template <int NQI>
__device__ __forceinline__ void stage_own_tile(const char* ks, const char* vs, int64_t srow, int r0, int S,
                                               uint8_t* slot, int q0) {
  const int lane = tix() & 63, rl = lane >> 4, pc = lane & 15;
  asm volatile("" ::: "memory");
#pragma unroll
  for (int qq = 0; qq < NQI; ++qq) {
    const int q = q0 + qq, r = 4 * q + rl;
    const int64_t off = (int64_t)(r0 + r < S ? r0 + r : 0) * srow + 16 * (pc ^ (r & 15));
    uint8_t* dst = slot + (q >> 2) * RSLOT + (q & 3) * 1024;
    load_lds16<true>(ks + off, dst);
    load_lds16<true>(vs + off, dst + 16 * DH * 2);
  }
}
template <int KT>
__device__ __forceinline__ void read_tile(const uint8_t* slot, const TileLanes<KT>& tl, RawTile<KT>& t) {
  if constexpr (KT == 0)
    read_tile_bf16(slot, tl, t);
  else
    read_tile_fp8(slot, tl, t);
}
// Ring geometry: slots per tile, tiles the ring holds.
template <int KT>
struct RingOf {
  static constexpr int spt = KT == 0 ? 2 : 1;
  static constexpr int tiles = RSLOTS / spt;
};

// The tiles of one unit for the agent's single query tile: wave w takes tiles w, w+4, ... of the unit's sequence,
// staged through its own LDS ring by direct loads (RingOf<KT>::tiles in flight): the cache tiles, then (last range
// only) the own-row tiles, which continue the same round robin.  In bf16 units the own-row tiles go through the
// ring like cache tiles (issued once the queries, keys and values of the head are published); in fp8 units they
// are bf16 while the cache tiles are not, and are read into registers after the cache tiles.  The waves' states
// are merged through LDS and written out (normalised if the agent has one range, else as the partial of this
// range).  Returns false if a wait failed.
template <int KT>
__device__ __forceinline__ bool attn_unit(const TickArgs& a, const TickParams& tp, const Dims& dm, int l,
                                          const AUnit& U, TickLds& L) {
  constexpr int TK = KT;  // tile kind of the cache tiles
  const int wave = tix() >> 6;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  // this wave's cache tiles: j = wave + 4 i, i < nc; then its own-row tiles j = first_own + 4 i, i < no
  const int nc = U.nct > wave ? (U.nct - wave + 3) / 4 : 0;
  const int first_own = (wave - U.nct % 4 + 4) % 4;
  const int no = KT == 0 && U.nst > first_own ? (U.nst - first_own + 3) / 4 : 0;
  const int n = nc + no;
  using RG = RingOf<KT>;
  uint8_t* lring = L.u.a.ring[wave][0];
  auto slot_of = [&](int i) { return lring + (i % RG::tiles) * RG::spt * RSLOT; };
  auto cache_tile = [&](int i) { return KT == 1 || i < nc; };  // fp8 units have no own-row tiles in the ring
  auto ctile = [&](int j) { return j + U.rot < U.nct ? j + U.rot : j + U.rot - U.nct; };  // streaming order
  auto row0 = [&](int i) { return cache_tile(i) ? U.i0 + 32 * ctile(wave + 4 * i) : 32 * (first_own + 4 * (i - nc)); };
  auto lim = [&](int i) { return cache_tile(i) ? U.i1 : tp.S; };
  auto ring_tile = [&](int i) {
    if (cache_tile(i))
      stage_tile<KT>(U.kc, U.vc, U.rsb, tp.start[U.b], a.cv.cap, U.i0, row0(i), U.i1, slot_of(i));
    else
      stage_own_tile<8>(U.ks, U.vs, (int64_t)dm.A * 2, row0(i), tp.S, slot_of(i), 0);
  };
  // The first tiles do not depend on this layer's projections: waves 0-2 issue them before waiting; wave 3 polls
  // the q, k and v column tiles of this head (its poll would otherwise return only after its own prefetch) and
  // issues its tiles afterwards.  Own-row tiles in the first places follow the wait.
  auto prefetch = [&]() {
#pragma unroll
    for (int dd = 0; dd < RG::tiles; ++dd)
      if (dd < nc) ring_tile(dd);
  };
  if (wave < 3) prefetch();
  const int RQ = row_blocks(tp.M);  // the flags of the head's q, k and v tiles, per row block
  if (!wg_wait(a.f_q + (int64_t)U.h * (DH / 16) * RQ * FPAD, 3 * (DH / 16) * RQ, st, a, L, DH / 16 * RQ, dm.A / 16 * RQ,
               3))
    return false;
  if (wave == 3) prefetch();
#pragma unroll
  for (int dd = 0; dd < RG::tiles; ++dd)
    if (dd >= nc && dd < n) ring_tile(dd);
  f32x4 o[1][8];
  float m_run[1] = {-INFINITY}, l_run[1] = {0.f};
#pragma unroll
  for (int k = 0; k < 8; ++k) o[0][k] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint4 qr[1][4];
  const TileLanes<TK> tl = tile_lanes<TK>();
  const int tt_one[1] = {0};
  load_q<1, KT == 1>(a, tp, dm, U.b, U.h, tt_one, 1, qr);
  auto qf = [&](int, int k) -> uint4 { return qr[0][k]; };
  // Pairs of tiles (i, i + 1) at ring places i % T, i % T + 1 (T = tiles the ring holds).  The pair is read once
  // every direct load this wave has issued has landed (no LDS read of this wave runs while its own direct loads
  // are in flight: reads in that window returned wrong values now and then); then the pair's places take tiles
  // i + T and i + T + 1, which stream in while the pair is computed.
#pragma unroll 1
  for (int i = 0; i < n; i += 2) {
    const bool two = i + 1 < n;
    vm_wait_all();
    RawTile<TK> ta, tb;
    read_tile<TK>(slot_of(i), tl, ta);
    if (two) read_tile<TK>(slot_of(i + 1), tl, tb);
    if (i + RG::tiles < n) ring_tile(i + RG::tiles);
    if (i + RG::tiles + 1 < n) ring_tile(i + RG::tiles + 1);
    if (two)
      tile_pair_compute<TK>(ta, tb, qr[0], row0(i), lim(i), row0(i + 1), lim(i + 1), U.ksc, o[0], m_run[0], l_run[0]);
    else
      tile_jobs<TK, 1, 1>(ta, qf, row0(i), lim(i), U.ksc, o, m_run, l_run);
  }
  if constexpr (KT == 1) {
    // fp8 values carry their scale: apply it to the cache part of the output before the own rows join
#pragma unroll
    for (int k = 0; k < 8; ++k) o[0][k] *= U.vsc;
    // own rows (bf16): tiles U.nct .. U.nct+nst-1 of the round robin
    if (U.nst > 0) {
      load_q<1, false>(a, tp, dm, U.b, U.h, tt_one, 1, qr);  // the queries again, as bf16
      for (int j = first_own; j < U.nst; j += 4) {
        RawTile<0> t;
        load_own_tile(U.ks, U.vs, (int64_t)dm.A * 2, 32 * j, tp.S, t);
        tile_jobs<0, 1, 1>(t, qf, 32 * j, tp.S, 1.f, o, m_run, l_run);
      }
    }
  }
  state_to_lds(state_of(L, wave), o[0], m_run[0], l_run[0]);
  __syncthreads();
  merge_states(a, tp, dm, U, 0, U.final_out, (int64_t)U.slot * tp.n_tt, L);
  __syncthreads();
  return true;
}


// One wave writes out a whole state from its LDS slots (rows [16][128], (m, l)[16]; see state_to_lds): lane l takes
// row l / 4, channels 32 (l % 4) .. + 31; normalised into the attention output if the agent has one range, else as
// the partial of item `item`.
__device__ __forceinline__ void write_state_rows(const TickArgs& a, const TickParams& tp, const Dims& dm, const AUnit& U,
                                                 int tt, int64_t item, const float* stw) {
  const int lane = tix() & 63, t = lane >> 2, c0 = (lane & 3) * 32;
  float4 v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = *reinterpret_cast<const float4*>(stw + t * 128 + c0 + 4 * i);
  const float m = stw[2048 + 2 * t], lt = stw[2048 + 2 * t + 1];
  if (U.final_out) {
    const int tok = tt * 16 + t;
    if (tok < tp.S) {
      const float f = 1.0f / lt;
      uint16_t* dst = a.attn + ((int64_t)U.b * tp.S + tok) * dm.A + (int64_t)U.h * DH + c0;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        st_loc16(dst + 8 * i, make_uint4(pack_bf16x2(v[2 * i].x * f, v[2 * i].y * f),
                                         pack_bf16x2(v[2 * i].z * f, v[2 * i].w * f),
                                         pack_bf16x2(v[2 * i + 1].x * f, v[2 * i + 1].y * f),
                                         pack_bf16x2(v[2 * i + 1].z * f, v[2 * i + 1].w * f)));
    }
  } else {
    float* po = a.att_o + (item * 16 + t) * 128 + c0;
#pragma unroll
    for (int i = 0; i < 8; ++i) st_loc_f4(po + 4 * i, v[i]);
    if ((lane & 3) == 0) {
      st_loc_f(a.att_ml + item * 32 + 2 * t, m);
      st_loc_f(a.att_ml + item * 32 + 2 * t + 1, lt);
    }
  }
}

// Many-query unit (query tiles tt0 .. tt0+nq-1, nq <= NQW = 6).  Wave 3 is the unit's loader: it stages every tile
// of the unit (cache tiles, then the own rows) into the workgroup ring of T tiles with direct loads, and never
// reads the ring; waves 0-2 only read the ring and compute (no wave reads LDS while its own direct loads are in
// flight: reads in that window returned wrong values now and then, so a wave that both loaded and computed could
// not overlap the two).  The ring holds two steps of G = T / 2 tiles: while the compute waves work on step k, the
// loader brings in step k + 1 and waits for it; a barrier then opens step k + 1 and frees step k's places.
//
// The compute waves split the arithmetic as jobs (query tile u, key class): a job takes the tiles i with
// i mod P = p (P = 1: the whole tile).  Per nq, with at most two jobs per wave w (w < 3):
//   1: tile 0, P = 3, p = w            2: tiles 0 and 1, P = 3, p = w        3: tile w whole
//   4: tile w whole; tile 3, P = 3, p = w                                    6: tiles w and w + 3 whole
//   5: tile w whole; tile 3, P = 2, p = w for w < 2; tile 4 whole for w = 2
// A whole job's state is written out by its wave; the key-split tiles are merged through LDS, one query tile at a
// time.  Output: normalised if the agent has one range, else the partial of this range.
template <int KT>
struct WRingOf {
  static constexpr int tb = KT == 0 ? 2 * RSLOT : RSLOT;  // bytes of a staged tile
  static constexpr int tiles = 4 * RSLOTS * RSLOT / tb;    // 8 (bf16) or 16 (fp8)
  static constexpr int own = 4 * RSLOTS * RSLOT / (2 * RSLOT);  // bf16 own-row tiles the ring holds
};
template <int KT>
__device__ __forceinline__ bool attn_unit_mq(const TickArgs& a, const TickParams& tp, const Dims& dm, int l,
                                             const AUnit& U, int tt0, int nq, TickLds& L) {
  using WR = WRingOf<KT>;
  constexpr int TK = KT;  // tile kind of the cache tiles
  constexpr int OK = 0;   // tile kind of the own rows (bf16)
  constexpr int G = WR::tiles / 2;  // tiles per step
  const int wave = tix() >> 6;
  const bool loader = wave == 3;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const int nc = U.nct;
  // this wave's jobs: query tile ju[j] (relative to tt0), key class p = jk[j] of jP[j]
  int nj = 0, ju[2] = {0, 0}, jP[2] = {1, 1}, jk[2] = {0, 0};
  auto add_job = [&](int u, int P, int pk) {
    ju[nj] = u;
    jP[nj] = P;
    jk[nj] = pk;
    ++nj;
  };
  if (!loader) {
    if (nq <= 2) {
      add_job(0, 3, wave);
      if (nq == 2) add_job(1, 3, wave);
    } else if (nq == 5) {
      add_job(wave, 1, 0);
      if (wave < 2) add_job(3, 2, wave);
      else add_job(4, 1, 0);
    } else {
      add_job(wave, 1, 0);
      if (nq == 4) add_job(3, 3, wave);
      if (nq == 6) add_job(wave + 3, 1, 0);
    }
  }
  // the key-split query tiles [s_lo, s_hi)
  const int s_lo = nq <= 2 ? 0 : 3, s_hi = nq <= 2 ? nq : (nq == 4 || nq == 5 ? 4 : 3);
  auto act_of = [&](int i) {
    return (nj > 0 && (jP[0] == 1 || i % jP[0] == jk[0]) ? 1 : 0) | (nj > 1 && (jP[1] == 1 || i % jP[1] == jk[1]) ? 2 : 0);
  };
  uint8_t* base = &L.u.a.ring[0][0][0];
  auto place = [&](int i) { return base + (i % WR::tiles) * WR::tb; };
  auto crow = [&](int i) { return U.i0 + 32 * (i + U.rot < nc ? i + U.rot : i + U.rot - nc); };  // i-th streamed
  auto stage = [&](int i) {  // the loader's loads of cache tile i (streaming order)
    if constexpr (KT == 0)
      stage_tile_bf16<8>(U.kc, U.vc, U.rsb, tp.start[U.b], a.cv.cap, U.i0, crow(i), U.i1, place(i), 0);
    else
      stage_tile_fp8<4>(U.kc, U.vc, U.rsb, tp.start[U.b], a.cv.cap, U.i0, crow(i), U.i1, place(i), 0);
  };
  // The first step's tiles do not depend on this layer's projections: the loader issues them before the wait, and
  // wave 0 (no loads in flight) polls the q, k and v column tiles of this head.
  if (loader)
    for (int i = 0; i < G && i < nc; ++i) stage(i);
  const int RQ = row_blocks(tp.M);  // the flags of the head's q, k and v tiles, per row block
  if (!wg_wait(a.f_q + (int64_t)U.h * (DH / 16) * RQ * FPAD, 3 * (DH / 16) * RQ, st, a, L, DH / 16 * RQ, dm.A / 16 * RQ,
               0)) {
    vm_wait_all();
    return false;
  }
  f32x4 o[2][8];
  float m_run[2], l_run[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
#pragma unroll
    for (int k = 0; k < 8; ++k) o[j][k] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[j] = -INFINITY;
    l_run[j] = 0.f;
  }
  const int tts[2] = {tt0 + ju[0], tt0 + ju[1]};
  uint4 qr[2][4];
  const TileLanes<TK> tl = tile_lanes<TK>();
  if (!loader) load_q<2, KT == 1>(a, tp, dm, U.b, U.h, tts, nj, qr);
  auto qf = [&](int j, int k) -> uint4 { return qr[j][k]; };
  // one step of the online softmax for the jobs that take tile i (index in its sequence)
  auto update = [&](auto kind, const auto& t, int i, int r0, int i1, float ksc) {
    constexpr int K = decltype(kind)::value;
    // the job sets that occur: {0} and {0, 1} (with two jobs, the second never runs without the first: they share
    // a key class, or the first takes the whole tile)
    const int act = act_of(i);
    if (act == 3)
      tile_jobs<K, 2, 3>(t, qf, r0, i1, ksc, o, m_run, l_run);
    else if (act == 1)
      tile_jobs<K, 2, 1>(t, qf, r0, i1, ksc, o, m_run, l_run);
  };
#pragma unroll 1
  for (int i = 0; i < nc; i += G) {
    if (loader) vm_wait_all();  // tiles i .. i + G - 1 have landed
    __syncthreads();            // and every compute wave is done with tiles i - G .. i - 1
    if (loader) {
      for (int e = 0; e < G; ++e)
        if (i + G + e < nc) stage(i + G + e);
    } else {
#pragma unroll 1
      for (int e = 0; e < G; ++e) {
        if (i + e < nc && act_of(i + e)) {
          RawTile<TK> t;
          read_tile<TK>(place(i + e), tl, t);
          update(std::integral_constant<int, TK>(), t, i + e, crow(i + e), U.i1, U.ksc);
        }
      }
    }
  }
  if (loader) vm_wait_all();
  if (KT == 1) {
    // fp8 values carry their scale: apply it to the cache part of the output before the own rows join
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int k = 0; k < 8; ++k) o[j][k] *= U.vsc;
  }
  // own rows (bf16), up to WR::own tiles per round through the ring
  for (int j0 = 0; j0 < U.nst; j0 += WR::own) {
    const int nown = min(WR::own, U.nst - j0);
    __syncthreads();  // every wave is done with the ring
    if (loader) {
      for (int j = 0; j < nown; ++j)
        stage_own_tile<8>(U.ks, U.vs, (int64_t)dm.A * 2, 32 * (j0 + j), tp.S, base + j * 2 * RSLOT, 0);
      vm_wait_all();
    } else if (KT == 1 && j0 == 0) {
      load_q<2, false>(a, tp, dm, U.b, U.h, tts, nj, qr);  // the queries as bf16
    }
    __syncthreads();
    if (!loader) {
      const TileLanes<OK> tlo = tile_lanes<OK>();
      for (int j = 0; j < nown; ++j) {
        if (act_of(j0 + j)) {
          RawTile<OK> t;
          read_tile<OK>(base + j * 2 * RSLOT, tlo, t);
          update(std::integral_constant<int, OK>(), t, j0 + j, 32 * (j0 + j), tp.S, 1.f);
        }
      }
    }
  }
  // whole jobs: each state goes through this wave's LDS slots into row order
  __syncthreads();  // every wave is done with the ring
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (j < nj && jP[j] == 1) {
      float* stw = state_of(L, wave);
      state_to_lds(stw, o[j], m_run[j], l_run[j]);
      write_state_rows(a, tp, dm, U, tt0 + ju[j], (int64_t)U.slot * tp.n_tt + tt0 + ju[j], stw);
    }
  }
  // key-split query tiles: each wave's state (empty if it has no job on the tile), merged in LDS
  for (int u = s_lo; u < s_hi; ++u) {
    __syncthreads();  // the ring (and the previous merge) is free
    f32x4 oe[8];
    float me = -INFINITY, le = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) oe[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (nj > 0 && jP[0] != 1 && ju[0] == u) {
#pragma unroll
      for (int k = 0; k < 8; ++k) oe[k] = o[0][k];
      me = m_run[0];
      le = l_run[0];
    } else if (nj > 1 && jP[1] != 1 && ju[1] == u) {
#pragma unroll
      for (int k = 0; k < 8; ++k) oe[k] = o[1][k];
      me = m_run[1];
      le = l_run[1];
    }
    state_to_lds(state_of(L, wave), oe, me, le);
    __syncthreads();
    merge_states(a, tp, dm, U, tt0 + u, U.final_out, (int64_t)U.slot * tp.n_tt + tt0 + u, L);
  }
  __syncthreads();  // the ring is free for the next unit
  return true;
}

// Attention work of XCD X: the segments (local head, agent) laid end to end, head-major (the short segments of
// ragged agents then fall into different slices), each weighing SEG_COST work units for its start-up (loading the
// queries and the first tiles, merging the waves' states) followed by one unit per 32-row cache tile and one per
// 32-row tile of the expert's own rows.  The slice that holds a segment's first own-row unit takes all its own rows
// (a later slice that holds only own-row units of the segment leaves an empty partial).  With enough work every
// workgroup takes an equal run of work units (slice); a segment whose tiles fall into several slices leaves one
// partial state per slice, merged afterwards by separate items (agent, head, query tile) in a fixed order.  With
// little work (fewer than about 4 cache tiles per workgroup) and few segments, workgroup s takes segment s whole and
// the others compute the projections (one agent of 32 heads: up to 992 cached rows).  Equal slices keep every
// workgroup streaming until the phase ends; the threshold is where the two plans measured equal (one agent, 32
// heads, 8 XCDs of 32 workgroups).
// Many-query units weigh no extra start-up: every slice pays one (its queries, its first group of tiles), and without
// the padding equal segments split into whole slices when the workgroups divide them evenly.
constexpr int SEG_COST = 24;
constexpr int SEG_COST_MQ = 0;
__device__ __forceinline__ bool attn_plan(const TickArgs& a, const TickParams& tp, const Dims& dm, TickLds& L) {
  const int X = uni(L.X), NX = uni(L.NX), n = uni(L.n);
  const int nh = head_lo(X + 1, NX, dm.H) - head_lo(X, NX, dm.H);
  const int nseg = tp.B * nh;  // <= NSEG = NTHR
  const int NT = nh * tp.seg_p[tp.B];  // work tiles (cache and own rows)
  const int mode = NT < 4 * n + nseg && nseg <= n ? 1 : 0;
  const int SC = tp.n_tt > 1 ? SEG_COST_MQ : SEG_COST;
  const int NC = NT + nseg * SC;  // work units
  const int g = tix();
  int np = 0;
  if (g < nseg) {
    const int j = g / tp.B, k = g % tp.B, w = tp.seg_w[k];
    const int g0 = j * (tp.seg_p[tp.B] + tp.B * SC) + tp.seg_p[k] + k * SC + SC;  // first tile's unit
    int sf = g;
    np = 1;
    if (mode == 0) {
      // slice of work unit c: the s with floor(s NC / n) <= c < floor((s + 1) NC / n)
      auto slice = [&](int c) { return (int)(((int64_t)(c + 1) * n - 1) / NC); };
      sf = slice(g0);
      np = slice(g0 + w - 1) - sf + 1;
    }
    L.seg0[g] = g0;
    L.segw[g] = w;
    L.sf[g] = (int16_t)sf;
    L.np[g] = (int16_t)np;
  }
  if (g == 0) {
    L.amode = mode;
    L.ant = NC;
  }
  // slots: exclusive prefix over segments of np where np > 1 (inclusive scan in LDS, then minus own)
  const int own = np > 1 ? np : 0;
  L.pb[g] = own;
  __syncthreads();
  for (int off = 1; off < NSEG; off <<= 1) {
    const int v = g >= off ? L.pb[g - off] : 0;
    __syncthreads();
    L.pb[g] += v;
    __syncthreads();
  }
  L.pb[g] -= own;
  __syncthreads();
  // the partial-state slots of this XCD must fit its tp.slot_x; a placement that breaks the host's bound fails the
  // tick (as a timed-out wait does) instead of writing past the range
  if (g == 0) {
    const int used = nseg > 0 ? L.pb[nseg - 1] + (L.np[nseg - 1] > 1 ? L.np[nseg - 1] : 0) : 0;
    L.ok = used <= tp.slot_x;
    if (!L.ok) st_dev(a.status, fail_tag(a));
  }
  __syncthreads();
  const bool ok = L.ok;
  __syncthreads();
  return ok;
}

template <int KT, bool MQ>
__device__ __forceinline__ bool phase_attn(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  constexpr int ES = KT == 0 ? 2 : 1;
  const int X = uni(L.X), s = uni(L.s), n = uni(L.n), NX = uni(L.NX);
  const int H = dm.H, A = dm.A, n_tt = tp.n_tt, B = tp.B;
  const int h0 = head_lo(X, NX, H), nh = head_lo(X + 1, NX, H) - h0;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const int nseg = B * nh, NC = uni(L.ant), mode = uni(L.amode);
  // this workgroup's work units [w0, w1)
  int w0, w1, g = 0;
  if (mode == 1) {
    w0 = s < nseg ? uni(L.seg0[s]) : 0;
    w1 = s < nseg ? w0 + uni(L.segw[s]) : 0;
    g = s;
  } else {
    w0 = (int)((int64_t)s * NC / n);
    w1 = (int)((int64_t)(s + 1) * NC / n);
    while (g < nseg && uni(L.seg0[g]) + uni(L.segw[g]) <= w0) ++g;
  }
  bool first = true;
  for (; w0 < w1 && g < nseg && uni(L.seg0[g]) < w1; ++g) {
    const int g0 = uni(L.seg0[g]), g1 = g0 + uni(L.segw[g]);
    const int t0 = max(w0, g0) - g0, t1 = min(w1, g1) - g0;  // the segment's units in this slice
    const int b = tp.order[g % B], h = h0 + g / B;
    const int npart = uni(L.np[g]);
    AUnit U;
    U.b = b;
    U.h = h;
    U.final_out = npart == 1;
    U.slot = X * tp.slot_x + uni(L.pb[g]) + (mode == 1 ? 0 : s - uni(L.sf[g]));
    const int cu = (tp.len[b] + 31) / 32;  // the segment's cache units; units cu .. are its own rows
    U.i0 = 32 * min(t0, cu);
    U.i1 = min(32 * min(t1, cu), tp.len[b]);
    U.nct = U.i1 > U.i0 ? (U.i1 - U.i0 + 31) / 32 : 0;
    U.nst = t0 <= cu && cu < t1 ? (tp.S + 31) / 32 : 0;  // the slice with the first own-row unit takes them all
    // Units that each take a whole (agent, head) start together at row 0 when the agents' lengths are equal, and
    // would stream addresses equal modulo the head's ring size: with a power-of-two ring the concurrent streams
    // then fall on few HBM channels (16 agents of 1,024 rows: 3,750 against 3,340 us with 1,040-row rings, with
    // some placements of the cache).  Such a unit starts at a tile of its own and wraps around.  Slices of a
    // longer range keep their order (they already start at different rows; rotating them was slower).
    U.rot = U.nct > 0 && U.i0 == 0 && U.i1 == tp.len[b] ? (int)((5u * (unsigned)h + 3u * (unsigned)b) % (unsigned)U.nct) : 0;
    const int64_t hb = cache_head_base(a.cv, b, l, h);  // ring slot 0 of (b, l, h)
    U.kc = (const char*)a.cv.k + hb * ES;
    U.vc = (const char*)a.cv.v + hb * ES;
    U.rsb = a.cv.rs * ES;
    U.ks = (const char*)a.kself + ((int64_t)b * tp.S * A + (int64_t)h * DH) * 2;
    U.vs = (const char*)a.vself + ((int64_t)b * tp.S * A + (int64_t)h * DH) * 2;
    U.ksc = U.vsc = 1.f;
    if (KT == 1) {
      const int64_t si = cache_scale_index(a.cv, b, l, h);
      U.ksc = a.cv.k_scale[si];
      U.vsc = a.cv.v_scale[si];
    }
    bool ok = true;
    if constexpr (!MQ) {
      ok = attn_unit<KT>(a, tp, dm, l, U, L);
    } else {
      for (int tt0 = 0; tt0 < n_tt && ok; tt0 += NQW)
        ok = attn_unit_mq<KT>(a, tp, dm, l, U, tt0, min(NQW, n_tt - tt0), L);
    }
    if (!ok) return false;
    if (first) TICK_SUB(l, 4);
    first = false;
    stores_done();
    __syncthreads();
    if (tix() == 0) {
      if (!U.final_out)
        st_loc(a.f_rng + (int64_t)U.slot * FPAD, st);
      else
        for (int tt = 0; tt < n_tt; ++tt) st_loc(a.f_attn + (((int64_t)b * H + h) * n_tt + tt) * FPAD, st);
    }
    __syncthreads();
  }
  // Merges of segments cut into several partials: item (segment, query tile) m on workgroup m mod n, after this
  // workgroup's own slice (slices never wait for merges, so these waits cannot form a cycle).
  for (int m = s; m < nseg * n_tt; m += n) {
    const int gm = m / n_tt, tt = m % n_tt;
    const int npart = uni(L.np[gm]);
    if (npart == 1) continue;
    const int b = tp.order[gm % B], h = h0 + gm / B;
    const int slot0 = X * tp.slot_x + uni(L.pb[gm]);
    if (!wg_wait(a.f_rng + (int64_t)slot0 * FPAD, npart, st, a, L)) return false;
    combine_ranges(a, tp, dm, b, h, slot0, npart, tt);
    stores_done();
    __syncthreads();
    if (tix() == 0) st_loc(a.f_attn + (((int64_t)b * H + h) * n_tt + tt) * FPAD, st);
    __syncthreads();
  }
  return true;
}

// ------------------------------------------------------------------------------------------ O
// The row-split projections (O, F1, D) work on items (column tile or unit k, row block r) of MTMAX*16 rows,
// item = k * R + r with R row blocks; workgroup s takes items s, s + n, ... (when n is a multiple of R, all of one
// workgroup's items share a row block, which it stages once).  With more than one row block this halves (or more)
// the rows a workgroup stages and multiplies, against every workgroup taking all rows of fewer tiles.

// Column tile k (of the residual) of the output projection over X's attention columns, rows of block r, as stamped
// partial words (reduced across the XCDs by phase_reduce).
__device__ __forceinline__ bool phase_oproj(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  const int X = uni(L.X), s = uni(L.s), n = uni(L.n), NX = uni(L.NX);
  const int d = dm.d, M = tp.M, A = dm.A, H = dm.H, nt = d / 16, R = row_blocks(M);
  const int h0 = head_lo(X, NX, H), nh = head_lo(X + 1, NX, H) - h0;
  const int kb0 = h0 * (DH / 32), nkb = nh * (DH / 32);  // <= 16
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const uint32_t st32 = (uint32_t)st;
  const LayerW W = layer_w(a, dm, l);
  uint64_t* po = a.po + (int64_t)X * nt * tp.Mp * 16;
  bool first = true;
  int staged = -1;  // row block in L.x
  const int total = nt * R;
  for (int it0 = s; it0 < total; it0 += IPF * n) {
    uint4 wg[IPF][4];
#pragma unroll
    for (int j = 0; j < IPF; ++j)
      if (it0 + j * n < total) load_unit_w(W.wo + (int64_t)((it0 + j * n) / R) * (A / 32) * WAVE, kb0, nkb, wg[j]);
    if (first && nh > 0 &&
        !wg_wait(a.f_attn + (int64_t)h0 * tp.n_tt * FPAD, tp.B * nh * tp.n_tt, st, a, L, nh * tp.n_tt, H * tp.n_tt))
      return false;
    if (first) TICK_SUB(l, 5);
#pragma unroll 1
    for (int j = 0; j < IPF && it0 + j * n < total; ++j) {
      const int item = it0 + j * n, k = item / R, r = item % R;
      uint4 w[4];
      pick_w(wg, j, w);
      const int m0 = r * MTMAX * 16, rows = min(MTMAX * 16, M - m0), mt_n = (rows + 15) / 16;
      if (nh > 0 && staged != r) stage(a.attn + h0 * DH, A, m0, rows, nh * DH, nullptr, 0, 0, 0.f, L);
      staged = r;
      unit_gemm(w, nkb, mt_n, L, [&](int mt, f32x4 sacc, int c, int grp) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = m0 + mt * 16 + 4 * grp + q;
          if (row < M)
            st_dev(po + ((int64_t)k * tp.Mp + row) * 16 + c, ((uint64_t)st32 << 32) | __float_as_uint(sacc[q]));
        }
      });
      if (first) TICK_SUB(l, 6);
      first = false;
    }
  }
  return true;
}

// ------------------------------------------------------------------------------------------ F1
// Items (unit k of X's FFN columns: 8 gate + 8 up rows of the packed matrix -> 8 SwiGLU outputs, row block r); the 4
// waves split K and reduce through LDS.  Each item publishes the flag f_z[unit * R + r].
__device__ __forceinline__ bool phase_gateup(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  const int X = uni(L.X), s = uni(L.s), n = uni(L.n), NX = uni(L.NX);
  const int d = dm.d, M = tp.M, F = dm.F, nt = d / 16, R = row_blocks(M);
  const int f0 = ffn_lo(X, NX, F), f1 = ffn_lo(X + 1, NX, F);
  const int u0 = f0 / 8, nu = (f1 - f0) / 8;
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const LayerW W = layer_w(a, dm, l);
  const uint16_t* xb = a.xb_mid;
  const float* ssq = a.ssq_mid;
  const int KB = d / 32;
  bool waited = false;
  int staged = -1;
  const int total = nu * R;
  for (int it0 = s; it0 < total; it0 += IPF * n) {
    uint4 wg[IPF][4];
#pragma unroll
    for (int j = 0; j < IPF; ++j)
      if (it0 + j * n < total) load_unit_w(W.wgu + (int64_t)(u0 + (it0 + j * n) / R) * KB * WAVE, 0, KB, wg[j]);
    if (!waited) {
      if (!wg_wait(a.f_mid, nt * tp.rblk, st, a, L)) return false;
      waited = true;
      TICK_SUB(l, 7);
    }
#pragma unroll 1
    for (int j = 0; j < IPF && it0 + j * n < total; ++j) {
      const int item = it0 + j * n, u = u0 + item / R, r = item % R;
      uint4 w[4];
      pick_w(wg, j, w);
      const int m0 = r * MTMAX * 16, rows = min(MTMAX * 16, M - m0), mt_n = (rows + 15) / 16;
      if (staged != r) stage(xb, d, m0, rows, d, ssq, tp.Ms, d, dm.eps, L);
      staged = r;
      unit_gemm(w, KB, mt_n, L, [&](int mt, f32x4 sacc, int c, int grp) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          sacc[q] *= L.r[mt * 16 + 4 * grp + q];  // RMSNorm row scale
          const float up = xor8(sacc[q]);
          const float gt = sacc[q];
          const float zz = gt / (1.0f + expf(-gt)) * up;
          const float zn = xor1(zz);
          const int row = m0 + mt * 16 + 4 * grp + q;
          if (c < 8 && (c & 1) == 0 && row < M)
            st_loc(reinterpret_cast<uint32_t*>(a.z + (int64_t)row * F + u * 8 + c), pack_bf16x2(zz, zn));
        }
      });
      if (item == s) TICK_SUB(l, 8);
      stores_done();
      __syncthreads();
      if (tix() == 0) st_loc(a.f_z + ((int64_t)u * R + r) * FPAD, st);
    }
  }
  return true;
}

// ------------------------------------------------------------------------------------------ D
// Items (column tile k, row block r) of the down projection over X's FFN columns, as stamped partial words (reduced
// across the XCDs by phase_reduce into the layer output).
__device__ __forceinline__ bool phase_down(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, TickLds& L) {
  const int X = uni(L.X), s = uni(L.s), n = uni(L.n), NX = uni(L.NX);
  const int d = dm.d, M = tp.M, F = dm.F, nt = d / 16, R = row_blocks(M);
  const int f0 = ffn_lo(X, NX, F), f1 = ffn_lo(X + 1, NX, F);
  const int kb0 = f0 / 32, nkb = (f1 - f0) / 32;  // <= 16
  const uint64_t st = stamp_of(a, l, dm.n_layers);
  const uint32_t st32 = (uint32_t)st;
  const LayerW W = layer_w(a, dm, l);
  uint64_t* pd = a.pd + (int64_t)X * nt * tp.Mp * 16;
  bool waited = false;
  int staged = -1;
  const int total = nt * R;
  for (int it0 = s; it0 < total; it0 += IPF * n) {
    uint4 wg[IPF][4];
#pragma unroll
    for (int j = 0; j < IPF; ++j)
      if (it0 + j * n < total) load_unit_w(W.wd + (int64_t)((it0 + j * n) / R) * (F / 32) * WAVE, kb0, nkb, wg[j]);
    if (!waited && nkb > 0 && !wg_wait(a.f_z + (int64_t)(f0 / 8) * R * FPAD, (f1 - f0) / 8 * R, st, a, L))
      return false;
    if (!waited) TICK_SUB(l, 9);
    waited = true;
#pragma unroll 1
    for (int j = 0; j < IPF && it0 + j * n < total; ++j) {
      const int item = it0 + j * n, k = item / R, r = item % R;
      uint4 w[4];
      pick_w(wg, j, w);
      const int m0 = r * MTMAX * 16, rows = min(MTMAX * 16, M - m0), mt_n = (rows + 15) / 16;
      if (nkb > 0 && staged != r) stage(a.z + f0, F, m0, rows, f1 - f0, nullptr, 0, 0, 0.f, L);
      staged = r;
      unit_gemm(w, nkb, mt_n, L, [&](int mt, f32x4 sacc, int c, int grp) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = m0 + mt * 16 + 4 * grp + q;
          if (row < M)
            st_dev(pd + ((int64_t)k * tp.Mp + row) * 16 + c, ((uint64_t)st32 << 32) | __float_as_uint(sacc[q]));
        }
      });
      if (item == s) TICK_SUB(l, 10);
    }
  }
  return true;
}

// ------------------------------------------------------------------------------------------ R1, R2
// The reduction across XCDs after the output projection (R1, second = false: into the FFN's input) or the down
// projection (R2: into the layer's output): every piece this workgroup owns (slot q mod n).  One call site in the
// layer loop, so the kernel holds one copy of this code.
__device__ __forceinline__ bool phase_reduce(const TickArgs& a, const TickParams& tp, const Dims& dm, int l, bool second,
                                             TickLds& L) {
  const int X = uni(L.X), s = uni(L.s), n = uni(L.n), NX = uni(L.NX), nt = dm.d / 16;
  const int t0 = tile_lo(X, NX, nt), t1 = tile_lo(X + 1, NX, nt);
  const uint64_t* part = second ? a.pd : a.po;
  uint16_t* xb = second ? a.xb_out : a.xb_mid;
  float* ssq = second ? a.ssq_out : a.ssq_mid;
  uint64_t* flag = second ? a.f_out : a.f_mid;
  float* hidden_l = second && a.hidden ? a.hidden + (int64_t)l * tp.M * dm.d : nullptr;
  for (int q = s; q < (t1 - t0) * tp.rblk; q += n)
    if (!reduce_piece(a, tp, dm, l, t0 + q / tp.rblk, q % tp.rblk, part, xb, ssq, flag, hidden_l, L)) return false;
  return true;
}

// ------------------------------------------------------------------------------------------ head
// wp[b] = mean over t < T of RMSNorm(h[b][t]) * g_final, times W_head^T, on the workgroups of XCD rank 0
// (agent b on slot b mod n0), from the residual once every piece of the last layer is published.  Thread tid
// owns columns tid and tid + 256 and holds the pooled rows in registers (16 rows per pass).
// Every workgroup that gave up (its failure is in the status word before it gets here) stores NaN into ALL
// waypoints, after its status store has completed.  The head workgroups store valid waypoints, wait for those
// stores, then read the status word and store NaN if a failure is recorded.  Either the head sees the failure, or
// the failing workgroup's status store (and so its NaN stores, which follow it) comes after the head's valid
// stores: the waypoints of a failed tick end as NaN in both orders.
__device__ __forceinline__ void poison_waypoints(const TickArgs& a, const TickParams& tp, const Dims& dm) {
  stores_done();
  __syncthreads();
  for (int i = tix(); i < tp.B * dm.n_out; i += NTHR) st_dev_f(a.waypoints + i, __builtin_nanf(""));
  stores_done();
}
__device__ __forceinline__ void phase_head(const TickArgs& a, const TickParams& tp, const Dims& dm, bool ok, TickLds& L) {
  const int d = dm.d, nl = dm.n_layers, T = tp.T;
  const int tid = tix(), wave = tid >> 6, lane = tid & 63;
  if (!ok) {
    poison_waypoints(a, tp, dm);
    return;
  }
  if (uni(L.X) != 0) return;
  const int s = uni(L.s), n = uni(L.n0);
  // Thread tid's two columns (n0, n1) of the head weights for every output, and their final gains: independent of
  // the last layer, so loaded before the wait, all at once (loaded one per step of the product they were as many
  // dependent memory round trips as the product has steps)
  constexpr int HO_MAX = 16;
  const bool regs = dm.n_out <= HO_MAX && s < tp.B;
  float hw0[HO_MAX], hw1[HO_MAX], g0 = 0.f, g1 = 0.f;
  if (regs && dm.head_kind != 1) {
    // every load unconditional (indices clamped in range, the unused values zeroed afterwards) and the dtype branch
    // outside the loop, so the loads issue back to back and cost one round trip
    const int no = dm.n_out, c0 = tid < d ? tid : d - 1, c1 = tid + NTHR < d ? tid + NTHR : d - 1;
    const bool in0 = tid < d, in1 = tid + NTHR < d;
    if (a.head_dtype == FSX_BF16) {
      const uint16_t* hw = reinterpret_cast<const uint16_t*>(a.head_w);
      uint16_t r0[HO_MAX], r1[HO_MAX];
#pragma unroll
      for (int o = 0; o < HO_MAX; ++o) {
        const int64_t row = (int64_t)(o < no ? o : no - 1) * d;
        r0[o] = hw[row + c0];
        r1[o] = hw[row + c1];
      }
#pragma unroll
      for (int o = 0; o < HO_MAX; ++o) {
        hw0[o] = o < no && in0 ? bf16_to_f32(r0[o]) : 0.f;
        hw1[o] = o < no && in1 ? bf16_to_f32(r1[o]) : 0.f;
      }
    } else {
      const float* hw = reinterpret_cast<const float*>(a.head_w);
#pragma unroll
      for (int o = 0; o < HO_MAX; ++o) {
        const int64_t row = (int64_t)(o < no ? o : no - 1) * d;
        hw0[o] = hw[row + c0];
        hw1[o] = hw[row + c1];
      }
#pragma unroll
      for (int o = 0; o < HO_MAX; ++o) {
        hw0[o] = o < no && in0 ? hw0[o] : 0.f;
        hw1[o] = o < no && in1 ? hw1[o] : 0.f;
      }
    }
    g0 = a.final_norm[c0];
    g1 = a.final_norm[c1];
    g0 = in0 ? g0 : 0.f;
    g1 = in1 ? g1 : 0.f;
  }
  for (int b = s; b < tp.B; b += n) {
    ok = wg_wait(a.f_out, d / 16 * tp.rblk, stamp_of(a, nl - 1, nl), a, L);  // every piece of the last layer
    if (!ok) {
      poison_waypoints(a, tp, dm);
      return;
    }
    const float* h = a.hres;  // tile-major [d/16][Mp][16]
    if (dm.head_kind == 1) {
      query_head_wg([&](int t, int col) { return ld_dev_f(h + ((int64_t)(col >> 4) * tp.Mp + b * tp.S + t) * 16 + (col & 15)); },
                    T, dm.n_out / 2, d, dm.eps, a.final_norm, a.qhead,
                    [&](int o, float v) { st_dev_f(a.waypoints + (int64_t)b * dm.n_out + o, v); },
                    reinterpret_cast<float*>(&L.u));
      continue;
    }
    const int n0 = tid, n1 = tid + NTHR;
    auto hv = [&](int m, int col) { return ld_dev_f(h + ((int64_t)(col >> 4) * tp.Mp + m) * 16 + (col & 15)); };
    float xm0 = 0.f, xm1 = 0.f;
    for (int t0 = 0; t0 < T; t0 += 16) {
      float v0[16], v1[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const bool in = t0 + t < T;
        const int m = b * tp.S + t0 + t;
        v0[t] = in && n0 < d ? hv(m, n0) : 0.f;
        v1[t] = in && n1 < d ? hv(m, n1) : 0.f;
      }
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        float sq = v0[t] * v0[t] + v1[t] * v1[t];
        sq = wave_sum(sq);
        if (lane == 0) L.red2[wave][t] = sq;
      }
      __syncthreads();
      if (tid < 16) {
        float sq = 0.f;
        for (int w = 0; w < NTHR / WAVE; ++w) sq += L.red2[w][tid];
        L.hr[tid] = 1.0f / sqrtf(sq / (float)d + dm.eps);
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
    if (regs) {
      // the pooled row's two columns of this thread times its weights, summed per wave, then over the 4 waves
      const float x0 = xm0 * g0 / (float)T, x1 = xm1 * g1 / (float)T;
#pragma unroll
      for (int o = 0; o < HO_MAX; ++o) {
        if (o < dm.n_out) {
          const float p = wave_sum(x0 * hw0[o] + x1 * hw1[o]);
          if (lane == 0) L.red2[wave][o] = p;
        }
      }
      __syncthreads();
      if (tid < dm.n_out) {
        float acc = 0.f;
        for (int w = 0; w < NTHR / WAVE; ++w) acc += L.red2[w][tid];
        st_dev_f(a.waypoints + (int64_t)b * dm.n_out + tid, acc);
      }
      __syncthreads();
      continue;
    }
    float* xm = L.tmp;
    if (n0 < d) xm[n0] = xm0 * a.final_norm[n0] / (float)T;
    if (n1 < d) xm[n1] = xm1 * a.final_norm[n1] / (float)T;
    __syncthreads();
    for (int o = wave; o < dm.n_out; o += NTHR / WAVE) {
      float acc = 0.f;
      for (int c = lane; c < d; c += WAVE) {
        const float wv = a.head_dtype == FSX_BF16 ? bf16_to_f32(((const uint16_t*)a.head_w)[(int64_t)o * d + c])
                                                 : ((const float*)a.head_w)[(int64_t)o * d + c];
        acc += xm[c] * wv;
      }
      acc = wave_sum(acc);
      if (lane == 0) st_dev_f(a.waypoints + (int64_t)b * dm.n_out + o, acc);
    }
    __syncthreads();
  }
  if (s >= tp.B) return;
  stores_done();
  __syncthreads();
  if (tix() == 0) L.ok = ld_dev(a.status) != fail_tag(a);  // one read, so the branch below is uniform
  __syncthreads();
  if (!L.ok) poison_waypoints(a, tp, dm);
}

// ------------------------------------------------------------------------------------------ kernel
// KT: cache element type (0 bf16, 1 fp8); MQ: more than one query tile per agent (S > 16).  Four instances, so that
// each carries only the attention variant it runs (smaller code for the instruction cache).
template <int KT, bool MQ>
__global__ __launch_bounds__(NTHR, 1) void k_tick(TickArgs a, TickParams tp, Dims dm) {
  __shared__ TickLds L;
  const int nl = dm.n_layers;
  trace_mark(a, 0, nl);
  bool ok = xcd_register(a, L);
  if (ok) ok = attn_plan(a, tp, dm, L);
  if (ok) phase_embed(a, tp, dm, L);
  trace_mark(a, 1, nl);
  for (int l = 0; l < nl && ok; ++l) {
    ok = phase_qkv(a, tp, dm, l, L);
    trace_mark(a, 2 + 16 * l, nl);
    ok = ok && phase_attn<KT, MQ>(a, tp, dm, l, L);
    trace_mark(a, 3 + 16 * l, nl);
    // O + R1, then F1, D + R2: the two reductions share one copy of their code (a loop of two passes)
#pragma unroll 1
    for (int second = 0; second < 2 && ok; ++second) {
      if (!second) {
        ok = phase_oproj(a, tp, dm, l, L);
      } else {
        ok = phase_gateup(a, tp, dm, l, L);
        trace_mark(a, 5 + 16 * l, nl);
        ok = ok && phase_down(a, tp, dm, l, L);
      }
      ok = ok && phase_reduce(a, tp, dm, l, second != 0, L);
      trace_mark(a, (second ? 6 : 4) + 16 * l, nl);
    }
  }
  phase_head(a, tp, dm, ok, L);
  trace_mark(a, 2 + 16 * nl, nl);
}

static const void* tick_fn(int kt, bool mq) {
  if (kt == 0) return mq ? (const void*)k_tick<0, true> : (const void*)k_tick<0, false>;
  return mq ? (const void*)k_tick<1, true> : (const void*)k_tick<1, false>;
}

hipError_t tick_occupancy(int kt, int* blocks_per_cu) {
  // every instance must fit
  int lo = 1 << 30;
  for (int mq = 0; mq < 2; ++mq) {
    int b = 0;
    const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, tick_fn(kt, mq != 0), NTHR, 0);
    if (e != hipSuccess) return e;
    lo = b < lo ? b : lo;
  }
  *blocks_per_cu = lo;
  return hipSuccess;
}

hipError_t launch_tick(const TickArgs& a, const TickParams& tp, const Dims& dm, int grid, hipStream_t s) {
  void* args[] = {(void*)&a, (void*)&tp, (void*)&dm};
  const void* f = tick_fn(a.cv.dtype == FSX_FP8_E4M3 ? 1 : 0, tp.n_tt > 1);
  return hipLaunchCooperativeKernel(f, dim3(grid), dim3(NTHR), args, 0, s);
}

__global__ void k_probe_xcds(uint32_t* out) {
  if (threadIdx.x == 0) out[blockIdx.x] = hw_xcc_id();
}

hipError_t probe_xcds(uint32_t* dev_out, int grid, hipStream_t s) {
  void* args[] = {(void*)&dev_out};
  return hipLaunchCooperativeKernel((const void*)k_probe_xcds, dim3(grid), dim3(64), args, 0, s);
}

}  // namespace fsx
