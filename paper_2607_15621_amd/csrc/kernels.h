// Host-visible launch interface of the expert-tick kernels (internal to libfsx).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/fsx.h"

namespace fsx {

// Per-forward description of the agents, passed by value in kernel arguments.
struct TickParams {
  int32_t B, S, T, M;                         // agents, tokens per agent, pooled tokens, rows = B*S
  int32_t n_tt;                               // ceil(S / 16): query tiles per (agent, head)
  int32_t chunk_rows;                         // per-phase path: cache rows per attention work item
  int32_t n_items;                            // per-phase path: attention work items
  int32_t Mp;                                 // M rounded up to 8: rows of tile-major activations
  int32_t Ms;                                 // M rounded up to 32: rows of the sums of squares
  int32_t n_units;                            // tick kernel: attention units
  int64_t pos[FSX_MAX_BATCH];                 // rotary position of token 0
  int64_t start[FSX_MAX_BATCH];               // ring slot of the oldest valid row
  int32_t len[FSX_MAX_BATCH];                 // valid cache rows
  int32_t chunk_prefix[FSX_MAX_BATCH + 1];    // per-phase path: chunk slots before agent b (ceil(len/chunk_rows) + 1 each)
  // tick kernel: attention units are (agent, range of range_rows[b] rows, head); agent b owns range slots
  // range_prefix[b] .. range_prefix[b+1]-1 (at least one, the last also holds the expert's own rows).  Units are
  // numbered agent by agent in the order order[0..B-1]; the k-th agent's units start at unit_prefix[k].
  int32_t range_prefix[FSX_MAX_BATCH + 1];
  int32_t range_rows[FSX_MAX_BATCH];
  int32_t unit_prefix[FSX_MAX_BATCH + 1];
  int32_t order[FSX_MAX_BATCH];
};

// Cache view of one layer.
struct CacheView {
  const void* k;     // base of the whole cache tensor
  const void* v;
  const float* k_scale;  // fp8 only: [batch][n_layers][H]
  const float* v_scale;
  int64_t cap;           // ring rows
  int32_t n_layers;
  int32_t layer;
  int32_t dtype;         // fsx_dtype
};

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
};

struct Dims {
  int d, H, Dh, A, F, n_layers, n_out;
  float eps, rope_base;
};

hipError_t launch_embed(const void* tokens, int tok_dtype, const float* g0, const TickParams& tp, const Dims& dm,
                        const Workspace& ws, hipStream_t s);
hipError_t launch_gemm_qkv(const FastWeights& w, const TickParams& tp, const Dims& dm, const Workspace& ws,
                           hipStream_t s);
hipError_t launch_attention(const CacheView& cv, const TickParams& tp, const Dims& dm, const Workspace& ws,
                            int waves_per_wg, hipStream_t s);
hipError_t launch_combine(const TickParams& tp, const Dims& dm, const Workspace& ws, hipStream_t s);
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

// ------------------------------------------------------------------ persistent tick kernel
struct TickLayer {
  const uint4* wqkv;
  const uint4* wo;
  const uint4* wgu;
  const uint4* wd;
  const float* attn_norm;
  const float* ffn_norm;
};

struct TickArgs {
  const TickLayer* layers;  // device [n_layers]
  const float* final_norm;
  const void* head_w;
  int head_dtype;
  int tok_dtype;
  const void* tokens;
  CacheView cv;
  float* waypoints;
  // exchanged inside the launch, device-coherent accesses
  float* q;
  uint16_t* kself;
  uint16_t* vself;
  float* att_o;
  float* att_ml;
  uint32_t* att_cnt;
  int n_att_cnt;
  float* part;
  uint32_t* o_cnt;
  uint32_t* d_cnt;
  uint32_t* sched;   // [n_layers] attention units taken beyond the first G
  // written once per launch (per layer); "tile-major" = [column tile][Mp rows][16 columns]
  float* h0;
  uint16_t* hb0;     // [d/16][Mp][16] bf16 copy of h0, tile-major
  uint16_t* hbmid;   // [L][d/16][Mp][16] bf16 copy of hmid, tile-major
  uint16_t* hbout;   // [L][d/16][Mp][16] bf16 copy of hout, tile-major
  float* ssq0;     // [d/16][Ms] per-tile sums of squares of h0
  float* rope;     // [M][Dh/2][2] cos, sin
  float* hmid;     // [L][M][d]
  float* hout;     // [L][M][d] (the caller's hidden buffer when given)
  float* ssq_mid;  // [L][d/16][Ms]
  float* ssq_out;  // [L][d/16][Ms]
  uint16_t* attn;  // [L][M][A]
  uint16_t* z;     // [L][F/8][Mp][8] SwiGLU output, tile-major
  // flags (stamps) and status
  uint64_t* f_embed;
  uint64_t* f_qkv;
  uint64_t* f_attn;
  uint64_t* f_hmid;
  uint64_t* f_z;
  uint64_t* f_hout;
  uint64_t* status;
  uint64_t epoch;
  uint64_t timeout_ticks;  // real-time counter ticks (100 MHz)
  int ks_o, ks_d;
  uint64_t* trace;         // optional: [grid][trace_events(n_layers)] real-time stamps per workgroup
};

// per workgroup: start, after the embedding, 16 events per layer (5 phase ends, then 11 sub-phase marks), end
__host__ __device__ inline int trace_events(int n_layers) { return 2 + 16 * n_layers + 1; }

hipError_t tick_occupancy(int kt, int* blocks_per_cu);
hipError_t launch_tick(const TickArgs& a, const TickParams& tp, const Dims& dm, int grid, hipStream_t s);

// ------------------------------------------------------------------ cache append
hipError_t launch_append(const fsx_cache_desc& c, const void* k_rows, const void* v_rows, int n_rows,
                         const int64_t* dst_first_slot /* host [batch] */, hipStream_t s);

// ------------------------------------------------------------------ simple per-op path (any dtype)
struct GenericWeights {
  const void* wq; const void* wk; const void* wv; const void* wo;
  const void* wg; const void* wu; const void* wd;
  const float* attn_norm; const float* ffn_norm;
};
struct GenericWorkspace {
  float* h; float* x; float* q; float* k; float* v; float* attn; float* g; float* u; float* rope;
};
hipError_t generic_tick(const GenericWeights* layers, const float* final_norm, const void* head_w, int wdtype,
                        const void* tokens, const CacheView& cv0, const TickParams& tp, const Dims& dm,
                        const GenericWorkspace& ws, float* waypoints, float* hidden, hipStream_t s);

}  // namespace fsx
