// Host-visible launch interface of the expert-tick kernels (internal to libfsx).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/fsx.h"
#include "head_device.h"

namespace fsx {

// Per-forward description of the agents, passed by value in kernel arguments.
struct TickParams {
  int32_t B, S, T, M;                         // agents, tokens per agent, pooled tokens, rows = B*S
  int32_t n_tt;                               // ceil(S / 16): query tiles per (agent, head)
  int32_t chunk_rows;                         // per-phase path: cache rows per attention work item
  int32_t n_items;                            // per-phase path: attention work items
  int32_t Mp;                                 // M rounded up to 8: rows of tile-major activations
  int32_t Ms;                                 // M rounded up to 32: rows of the sums of squares
  int64_t pos[FSX_MAX_BATCH];                 // rotary position of token 0
  int64_t start[FSX_MAX_BATCH];               // ring slot of the oldest valid row
  int32_t len[FSX_MAX_BATCH];                 // valid cache rows
  int32_t chunk_prefix[FSX_MAX_BATCH + 1];    // per-phase path: chunk slots before agent b (ceil(len/chunk_rows) + 1 each)
  // tick kernel attention: agents in the order order[0..B-1]; the k-th weighs seg_w[k] work tiles per head
  // (its 32-row cache tiles, then the 32-row tiles of the expert's own rows), seg_p[k] = seg_w[0] + ... +
  // seg_w[k-1]; partial-state slots of XCD X
  // are X * slot_x .. X * slot_x + slot_x - 1
  int32_t order[FSX_MAX_BATCH];
  int32_t seg_w[FSX_MAX_BATCH];
  int32_t seg_p[FSX_MAX_BATCH + 1];
  int32_t slot_x;
  // tick kernel: row blocks of every residual column tile in the cross-XCD reductions (pieces; see reduce_piece)
  int32_t rblk;
};

// Cache view of one layer.  Element offset of (agent b, layer l, head h, ring slot j, channel c):
// b * bs + l * H * cap * Dh + h * hs + j * rs + c, with (hs, rs) = (cap * Dh, Dh) for a head-major cache and
// (Dh, H * Dh) for a token-major one; bs = n_layers * H * cap * Dh, or 0 when every agent reads the same rings
// (a shared cache).  fp8 scale of (b, l, h): [b * sbs + l * H + h], sbs = n_layers * H or 0.
struct CacheView {
  const void* k;     // base of the whole cache tensor
  const void* v;
  const float* k_scale;  // fp8 only: [batch][n_layers][H] ([1][n_layers][H] when shared)
  const float* v_scale;
  int64_t cap;           // ring rows
  int64_t hs;            // elements between the rows of two heads of one slot
  int64_t rs;            // elements between two ring slots of one head
  int64_t bs;            // elements between the rings of two agents (0: shared)
  int32_t sbs;           // scales between two agents (0: shared)
  int32_t n_layers;
  int32_t layer;
  int32_t dtype;         // fsx_dtype
  int32_t H, Dh;
};
// Element offset of row slot 0 of (agent b, layer l, head h).
__host__ __device__ inline int64_t cache_head_base(const CacheView& cv, int b, int l, int h) {
  return (int64_t)b * cv.bs + (int64_t)l * cv.H * cv.cap * cv.Dh + (int64_t)h * cv.hs;
}
__host__ __device__ inline int64_t cache_scale_index(const CacheView& cv, int b, int l, int h) {
  return (int64_t)b * cv.sbs + (int64_t)l * cv.H + h;
}

// ------------------------------------------------------------------ packing (create time)
enum PackKind { PACK_PLAIN = 0, PACK_ROPE_PAIRS = 1, PACK_SWIGLU_PAIRS = 2 };
hipError_t launch_pack(const uint16_t* a, const uint16_t* b, int N, int K, int kind, int param, const float* gain,
                       void* dst, hipStream_t s);

// ------------------------------------------------------------------ fused-path phases
struct FastWeights {
  const uint4* wqkv;   // packed [3A][d]  (q, k rows paired for rotary)
  const uint4* wo;     // packed [d][A]
  const uint4* wgu;    // packed [2F][d]  (gate/up rows paired)
  const uint4* wd;     // packed [d][F]
  const float* attn_norm;
  const float* ffn_norm;
};

struct Workspace {
  float* h;          // [M][d] residual stream
  uint16_t* xb;      // [M][max(d, ...)] bf16 normalised input of the next projection
  float* q;          // [M][A] rotated, pre-scaled queries
  uint16_t* kself;   // [M][A] bf16 rotated keys of the expert tokens
  uint16_t* vself;   // [M][A] bf16 values of the expert tokens
  uint16_t* attn;    // [M][A] bf16 attention output
  uint16_t* z;       // [M][F] bf16 SwiGLU output
  float* part;       // [ksplit][M][d] split-K partial sums
  float* att_o;      // [items][16][Dh] unnormalised partial attention outputs
  float* att_ml;     // [items][16][2] running max (log2 units) and sum
  float* rope;       // [M][Dh/2][2] cos, sin
  float* ss;         // [M][d/512] per-chunk sums of squares (wide rows)
  float* rs;         // [M] RMSNorm scale of each row (wide rows)
  uint32_t* rcnt;    // [M] chunks of the row reduced so far (wide rows; zero between launches)
};

struct Dims {
  int d, H, Dh, A, F, n_layers, n_out;
  float eps, rope_base;
  int head_kind;  // 0: mean over the expert tokens + linear; 1: two-layer head over the waypoint queries
};

// Rows wide enough (the backbone's width) that the per-phase reductions split them into chunks of RN_CHUNK columns,
// one workgroup each, and leave the RMSNorm scale to the next projection.
constexpr int RN_CHUNK = 512;
__host__ __device__ inline bool wide_rows(const Dims& dm) { return dm.d >= 4 * RN_CHUNK && dm.d % RN_CHUNK == 0; }

hipError_t launch_embed(const void* tokens, int tok_dtype, const float* g0, const TickParams& tp, const Dims& dm,
                        const Workspace& ws, hipStream_t s);
// after_reduction: xb comes from a reduction (not from the embedding); for wide rows it is then unscaled and the
// projection applies the RMSNorm row scales from the chunk sums of squares.
hipError_t launch_gemm_qkv(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                           hipStream_t s, bool after_reduction);
hipError_t launch_attention(const CacheView& cv, const TickParams& tp, const Dims& dm, const Workspace& ws,
                            int waves_per_wg, hipStream_t s, bool causal = false);
// Merges the attention's partial states; with rows_into, the same launch also stores the layer's new rows
// (ws.kself / ws.vself, B agents x S tokens) into ring slots (start + len + t) mod capacity of cache layer
// rows_into->layer (after the attention has read the old rows).
hipError_t launch_combine(const TickParams& tp, const Dims& dm, const Workspace& ws, hipStream_t s,
                          const CacheView* rows_into = nullptr);
hipError_t launch_gemm_o(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                         int ksplit, hipStream_t s);
hipError_t launch_gemm_gu(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                          hipStream_t s);
hipError_t launch_gemm_down(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                            int ksplit, hipStream_t s);
hipError_t launch_reduce_norm(const TickParams& tp, const Dims& dm, const Workspace& ws, int ksplit,
                              const float* gain, float* hidden_layer, hipStream_t s);
hipError_t launch_head(const TickParams& tp, const Dims& dm, const Workspace& ws, const float* final_norm,
                       const void* head_w, int head_dtype, float* waypoints, hipStream_t s);
// The two-layer query head of every agent from a row-major residual h [M][d] (both per-op paths).
hipError_t launch_query_head(const float* h, const TickParams& tp, const Dims& dm, const float* final_norm,
                             const QueryHead& qh, float* waypoints, hipStream_t s);

// ------------------------------------------------------------------ persistent tick kernel
// The tick kernel splits every layer over the chip's XCDs the way a tensor-parallel layer is split over
// devices: XCD X owns a contiguous range of heads and of FFN columns.  Buffers marked "per XCD" hold one
// replica per XCD rank (at most NXMAX); those indexed by head or FFN unit are written and read by one XCD only;
// the residual and its bf16 copies are written once (each piece by one workgroup) and read by every XCD.
constexpr int NXMAX = 16;
constexpr int NXR = 8;      // XCDs the cross-XCD reductions read at most (the XCD count of gfx950 parts)
constexpr int FPAD = 16;     // flags are 64-bit stamps, one per 128-byte line (index * FPAD)
constexpr int XFLAGS = 512;  // flag slots per XCD of the per-XCD flag arrays

struct TickArgs {
  const char* wbase;   // packed weights of layer 0; layers follow back to back (see layer_w)
  const float* final_norm;
  const void* head_w;
  int head_dtype;
  QueryHead qhead;     // head kind 1
  int tok_dtype;
  const void* tokens;
  CacheView cv;
  float* waypoints;
  float* hidden;       // optional caller buffer [n_layers][M][d]
  uint64_t* reg;       // [grid] registration words: epoch << 8 | hardware XCD id
  // written by the owner of each piece, read by every XCD
  float* hres;         // residual stream, tile-major [d/16 column tiles][Mp rows][16 columns]
  uint16_t* xb_mid;    // [Mp][d] bf16 copy of the residual after attention (input of the FFN)
  uint16_t* xb_out;    // [Mp][d] bf16 copy of the residual after the FFN (input of the next layer)
  float* ssq_mid;      // [d/16][Ms] per-tile sums of squares
  float* ssq_out;
  // per XCD
  float* rope;         // [M][Dh/2][2] cos, sin
  int64_t x_stride_r;  // floats between replicas of rope
  // by head / FFN unit
  float* q;            // [M][A] rotated, pre-scaled queries
  uint16_t* kself;     // [M][A]
  uint16_t* vself;     // [M][A]
  uint16_t* attn;      // [M][A]
  uint16_t* z;         // [Mp][F] SwiGLU output
  float* att_o;        // [slot * n_tt + query tile][16][Dh] partial attention states
  float* att_ml;       // [slot * n_tt + query tile][16][2]
  // crossing XCDs: stamped 8-byte words (payload in the low half, stamp in the high half)
  uint64_t* po;        // [NXMAX][d/16][Mp][16] output-projection partials
  uint64_t* pd;        // [NXMAX][d/16][Mp][16] down-projection partials
  // flags (stamps), each in its own 128-byte line: element [i] lives at f[i * FPAD]
  uint64_t* f_rope;    // [NXMAX][XFLAGS] by workgroup slot
  uint64_t* f_out;     // [XFLAGS] by residual piece (column tile * rblk + row block)
  uint64_t* f_mid;     // [XFLAGS] by residual piece
  uint64_t* f_q;       // [3A/16][row blocks of 80 rows]
  uint64_t* f_attn;    // [B*H][n_tt] per query tile
  uint64_t* f_rng;     // [slot] partial states written
  uint64_t* f_z;       // [F/8][row blocks of 80 rows]
  uint64_t* status;
  uint64_t epoch;
  uint64_t timeout_ticks;  // real-time counter ticks (100 MHz)
  uint64_t* trace;         // optional: [grid][trace_events(n_layers)] real-time stamps per workgroup
};

// per workgroup: start, after the embedding, 16 events per layer (5 phase ends, then 11 sub-phase marks), end
__host__ __device__ inline int trace_events(int n_layers) { return 2 + 16 * n_layers + 1; }

hipError_t tick_occupancy(int kt, int* blocks_per_cu);
hipError_t launch_tick(const TickArgs& a, const TickParams& tp, const Dims& dm, int grid, hipStream_t s);
// Hardware XCD id of every workgroup of a one-workgroup-per-CU launch (create-time placement check).
hipError_t probe_xcds(uint32_t* dev_out, int grid, hipStream_t s);

// Zero `bytes` (a multiple of 256) at p with a kernel.
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);

// ------------------------------------------------------------------ measurement helper
// One read-only pass over `bytes` (a multiple of 16) of buf; mode 0 register loads, 1 direct loads into LDS;
// sink: DEVICE [1024] uint32 checksum words.
hipError_t launch_probe_read(const void* buf, int64_t bytes, int mode, uint32_t* sink, hipStream_t s);

// ------------------------------------------------------------------ cache append
hipError_t launch_append(const fsx_cache_desc& c, const void* k_rows, const void* v_rows, int n_rows,
                         const int64_t* dst_first_slot /* host [batch] */, hipStream_t s);
// bf16 / fp32 rows (rows_dtype) encoded into an fp8 cache with its existing scales.
hipError_t launch_append_quantize(const fsx_cache_desc& c, const void* k_rows, const void* v_rows, int rows_dtype,
                                  int n_rows, const int64_t* dst_first_slot, hipStream_t s);

// ------------------------------------------------------------------ simple per-op path (any dtype)
struct GenericWeights {
  const void* wq; const void* wk; const void* wv; const void* wo;
  const void* wg; const void* wu; const void* wd;
  const float* attn_norm; const float* ffn_norm;
};
struct GenericWorkspace {
  float* h; float* x; float* q; float* k; float* v; float* attn; float* g; float* u; float* rope;
};
hipError_t generic_tick(const GenericWeights* layers, const float* final_norm, const void* head_w,
                        const QueryHead& qhead, int wdtype,
                        const void* tokens, const CacheView& cv0, const TickParams& tp, const Dims& dm,
                        const GenericWorkspace& ws, float* waypoints, float* hidden, hipStream_t s);

}  // namespace fsx
