/*
 * fsx.h -- C ABI of the action-expert fast path (MI355X / gfx950).
 *
 * The method (Sec. 3.1, "Action Expert with Per-Layer Cache Attention"): a small
 * transformer (the "action expert") runs once per control tick.  At each of its
 * layers it projects its own tokens into the frozen backbone's attention geometry
 * (H heads of width Dh), attends jointly over [the backbone's cached keys/values
 * of that layer ; its own keys/values] (Eq. (1)), projects back to width d and
 * applies a SwiGLU block; a head regresses waypoints.  The backbone never attends
 * to expert tokens, so the cache is read-only for the expert and can be kept as
 * standing state that the slow system extends by appending rows every K ticks
 * (Sec. 3.3, "Asynchronous Deployment").
 *
 * This header exposes exactly that per-tick path:
 *   fsx_expert_create      -- pack the expert's weights into library-owned device memory
 *   fsx_expert_forward     -- one tick: all layers + head, for a batch of agents
 *   fsx_cache_append_rows  -- append new cached K/V rows (the slow system's output)
 * plus destroy / error / introspection helpers.
 *
 * Conventions shared by every call
 *   - All functions return an fsx_status (0 = FSX_OK).  Argument and shape checks
 *     run before any GPU work is enqueued; on error nothing is enqueued and
 *     fsx_last_error() (thread-local) holds a message.
 *   - "device" pointers are HIP device memory of the current device; "host"
 *     pointers are ordinary CPU memory.  No call keeps a caller pointer after it
 *     returns, except that enqueued GPU work reads/writes the caller's device
 *     buffers later in stream order.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Work is
 *     enqueued on it asynchronously; GPU faults surface at the caller's next
 *     synchronisation of that stream.
 *   - Matrices use the nn.Linear layout [out][in], row-major, densely packed.
 *   - No exception crosses this boundary.
 */
#ifndef FSX_H
#define FSX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FSX_OK = 0,
  FSX_E_INVALID = 1,     /* bad argument, NULL pointer, inconsistent shapes */
  FSX_E_UNSUPPORTED = 2, /* valid request the library does not implement */
  FSX_E_CAPACITY = 3,    /* batch/rows beyond what was provisioned, or ring full under FSX_APPEND_ERROR */
  FSX_E_OOM = 4,         /* device allocation failed */
  FSX_E_HIP = 5          /* a HIP runtime call or kernel launch failed */
} fsx_status;

typedef enum {
  FSX_F32 = 0,      /* IEEE binary32 */
  FSX_BF16 = 1,     /* bfloat16 */
  FSX_FP8_E4M3 = 2  /* OCP FP8 E4M3 ("e4m3fn": bias 7, max 448, no inf); cache only */
} fsx_dtype;

enum { FSX_APPEND_RING = 0, FSX_APPEND_ERROR = 1 };

/* Layouts of the cache tensors (fsx_cache_desc.layout): HEAD_MAJOR or TOKEN_MAJOR, optionally | SHARED. */
enum {
  FSX_CACHE_HEAD_MAJOR = 0,  /* [batch][n_layers][H][capacity][Dh]: one contiguous ring per (agent, layer, head) */
  FSX_CACHE_TOKEN_MAJOR = 1, /* [batch][n_layers][capacity][H][Dh]: one ring slot holds a cached token for every head */
  FSX_CACHE_SHARED = 2       /* flag: k, v (and fp8 scales) hold ONE agent's rings, which every agent of the batch
                                reads through its own start / len / pos -- the expert blocks of one training clip,
                                each seeing a different (stale) prefix of the same cache (Sec. 3.2) */
};

/* Flags of fsx_expert_cfg.flags. */
enum {
  FSX_FLAG_GENERIC = 1,     /* force the simple per-op kernels instead of the fused tick kernel */
  FSX_FLAG_MULTI_LAUNCH = 2, /* run the fused path as one launch per phase instead of one persistent launch */
  FSX_FLAG_TRACE = 4         /* tick kernel records per-workgroup phase timestamps (fsx_expert_trace) */
};

#define FSX_MAX_BATCH 64

/* Sizes of the expert (Sec. 3.1: 32 layers, width d = 512, backbone geometry 32 heads x 128,
 * 10 expert tokens, 5 (x, y) waypoints).  The FFN width is not given by the paper. */
typedef struct {
  int32_t n_layers;         /* > 0 */
  int32_t d_model;          /* d  (expert width) */
  int32_t n_heads;          /* H  (backbone heads) */
  int32_t head_dim;         /* Dh (backbone head width); A = H * Dh */
  int32_t d_ffn;            /* SwiGLU hidden width */
  int32_t n_expert_tokens;  /* T: tokens pooled by the waypoint head */
  int32_t n_out;            /* head outputs (10 = 5 waypoints x (x, y)) */
  int32_t max_batch;        /* agents per forward, 1..FSX_MAX_BATCH */
  int32_t max_frame_tokens; /* F: extra current-frame tokens per agent, >= 0 */
  int32_t dtype;            /* fsx_dtype of weights and tokens: FSX_F32 or FSX_BF16 */
  float rope_base;          /* rotary base for expert q/k (pairs j, j+Dh/2); 0 = no rotary */
  float rms_eps;            /* RMSNorm epsilon */
  int32_t flags;            /* FSX_FLAG_* */
  int32_t tick_timeout_us;  /* bound on any wait inside the tick kernel; 0 = 2 s */
  int32_t head_kind;        /* FSX_HEAD_MEAN_LINEAR or FSX_HEAD_QUERY_MLP */
  int32_t head_hidden;      /* FSX_HEAD_QUERY_MLP: width of the head's hidden layer, 1..2048; ignored otherwise */
} fsx_expert_cfg;

/* Waypoint heads (fsx_expert_cfg.head_kind). */
enum {
  FSX_HEAD_MEAN_LINEAR = 0, /* final RMSNorm, mean over the T expert tokens, Linear(d -> n_out) without bias */
  FSX_HEAD_QUERY_MLP = 1    /* the paper's head (Sec. 3.1): the last n_out / 2 expert tokens are waypoint queries,
                               each decoded to one (x, y) by final RMSNorm, Linear(d -> head_hidden) + bias, GELU
                               (erf form), Linear(head_hidden -> 2) + bias; n_out even, n_out / 2 <= min(T, 8) */
};

/* The head's parameters, DEVICE pointers; matrices in cfg.dtype, biases fp32. */
typedef struct {
  const void* w;    /* MEAN_LINEAR: [n_out][d]; QUERY_MLP: first layer [head_hidden][d] */
  const float* b;   /* QUERY_MLP: [head_hidden]; NULL for MEAN_LINEAR */
  const void* w2;   /* QUERY_MLP: second layer [2][head_hidden]; NULL for MEAN_LINEAR */
  const float* b2;  /* QUERY_MLP: [2]; NULL for MEAN_LINEAR */
} fsx_head_weights;

/* One layer's parameters, DEVICE pointers, elements of cfg.dtype (norm gains always fp32). */
typedef struct {
  const void* wq;          /* [A][d] */
  const void* wk;          /* [A][d] */
  const void* wv;          /* [A][d] */
  const void* wo;          /* [d][A] */
  const void* w_gate;      /* [d_ffn][d] */
  const void* w_up;        /* [d_ffn][d] */
  const void* w_down;      /* [d][d_ffn] */
  const float* attn_norm;  /* [d] RMSNorm gain before attention */
  const float* ffn_norm;   /* [d] RMSNorm gain before the FFN */
} fsx_layer_weights;

/* The backbone's per-layer KV cache for a batch of agents (Sec. 3.1: per layer the cache is L tokens of
 * H heads x Dh; Sec. 3.3: it is standing state that grows by appends).  Each (agent, layer) holds a ring of
 * `capacity` token slots; a slot holds one cached token's key (or value) for every head.  Two layouts of
 * the same ring are accepted (`layout`): head-major, where each (agent, layer, head) owns `capacity`
 * contiguous rows of Dh elements, and token-major, where a slot's H x Dh elements are contiguous (the
 * L x (H*Dh) rows of a backbone's cache).  Either way one head's row of one token is Dh contiguous
 * elements.  Keys are stored already rotated.  The valid rows of agent b are ring slots
 * (start[b] + i) mod capacity, i < len[b], the same slots in every layer and head. */
typedef struct {
  int32_t dtype;           /* FSX_F32 | FSX_BF16 | FSX_FP8_E4M3 */
  int32_t batch;           /* agents described by this descriptor */
  int32_t n_layers;        /* must equal the expert's */
  int32_t n_heads;         /* must equal the expert's */
  int32_t head_dim;        /* must equal the expert's */
  int32_t layout;          /* FSX_CACHE_HEAD_MAJOR (0) or FSX_CACHE_TOKEN_MAJOR (1), optionally | FSX_CACHE_SHARED;
                              FSX_E_INVALID otherwise */
  int64_t capacity;        /* ring slots per (agent, layer) */
  void* k;                 /* DEVICE [batch][n_layers][H][capacity][Dh] (head-major) or
                              [batch][n_layers][capacity][H][Dh] (token-major); batch = 1 in memory when shared */
  void* v;                 /* DEVICE, same layout */
  const float* k_scale;    /* FP8 only: DEVICE [batch][n_layers][H] ([1][n_layers][H] when shared), stored value =
                              code * scale */
  const float* v_scale;    /* FP8 only: DEVICE, as k_scale */
  int64_t* start;          /* HOST [batch]: ring slot of the oldest valid row */
  int64_t* len;            /* HOST [batch]: valid rows, 0..capacity */
  int64_t* pos;            /* HOST [batch]: position of the agent's expert token 0 (rotary angle) */
} fsx_cache_desc;

typedef struct fsx_expert fsx_expert;

/* Pack an expert's weights into library-owned device memory.
 *   cfg        sizes and dtype (validated; FSX_E_INVALID / FSX_E_UNSUPPORTED on bad values)
 *   layers     HOST array of cfg.n_layers descriptors (DEVICE weight pointers)
 *   final_norm DEVICE [d] fp32 gain of the RMSNorm before the head
 *   head       HOST struct of DEVICE pointers to the head's parameters (cfg.head_kind)
 *   stream     used for the packing copies; the call synchronises it before returning,
 *              so the caller may free its weight buffers afterwards
 *   out        receives the handle (NULL on failure)
 * Allocates the packed weights and a workspace sized for cfg.max_batch agents of
 * T + max_frame_tokens tokens. */
int fsx_expert_create(const fsx_expert_cfg* cfg, const fsx_layer_weights* layers, const float* final_norm,
                      const fsx_head_weights* head, void* stream, fsx_expert** out);

/* One control tick for `batch` agents (Sec. 3.1, Eq. (1); Sec. 3.3: the expert reads the cache as-is).
 *   cache          descriptor; only rows (start+i) mod capacity, i < len[b], are read.  The
 *                  cache is never written.  batch <= cache->batch.
 *   tokens         DEVICE [batch][S][d] (cfg.dtype), S = T + n_frame_tokens; rows < T are the
 *                  expert tokens, the rest current-frame tokens.  Token t of agent b sits at
 *                  rotary position pos[b] + t.
 *   n_frame_tokens 0..cfg.max_frame_tokens
 *   waypoints      DEVICE [batch][n_out] fp32 output
 *   hidden         DEVICE [n_layers][batch][S][d] fp32 output of every layer, or NULL
 * Uses only library-owned workspace; allocates nothing.  Calls that overlap on one
 * expert handle (e.g. from two streams) race on its workspace. */
int fsx_expert_forward(fsx_expert* ex, const fsx_cache_desc* cache, const void* tokens, int32_t batch,
                       int32_t n_frame_tokens, float* waypoints, float* hidden, void* stream);

/* The same tick as fsx_expert_forward, for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): it allocates nothing, neither in the call nor
 * through the handle's workspace.  The tick kernel's workspace lives in a static device array of the library of
 * 48 MiB per device (held until the process ends; its device address is looked up on the first call on a device).
 * Each call first clears the part of that array that must start at zero, with a kernel on `stream`, so a call does
 * not depend on what an earlier call left there; calls that overlap on one device (other streams or threads) race
 * on the array and must be serialised by the caller.  Arguments and results as fsx_expert_forward.
 *   FSX_E_CAPACITY    the call's sizes need more than the array holds (the message gives the bytes needed;
 *                     e.g. 16 agents x 10 tokens or one agent x 74 tokens fit, 64 agents do not)
 *   FSX_E_UNSUPPORTED the handle does not run the persistent tick kernel (fp32 weights, FSX_FLAG_GENERIC,
 *                     FSX_FLAG_MULTI_LAUNCH, shapes outside the per-XCD split)
 * A tick that gives up on a wait writes NaN waypoints; fsx_expert_status does not report calls made here. */
int fsx_expert_forward_noalloc(fsx_expert* ex, const fsx_cache_desc* cache, const void* tokens, int32_t batch,
                               int32_t n_frame_tokens, float* waypoints, float* hidden, void* stream);

/* Append n_rows new cached rows to every (agent, layer, head) of the cache (Sec. 3.3: every K ticks
 * the slow system appends the current frame's tokens through an incremental forward).
 *   k_rows, v_rows DEVICE, in the cache's layout with n_rows slots: [cache->batch][n_layers][H][n_rows][Dh]
 *                  for a head-major cache, [cache->batch][n_layers][n_rows][H][Dh] for a token-major one;
 *                  elements of cache->dtype (fp8: codes already scaled by the cache's k_scale / v_scale);
 *                  Dh elements must be a multiple of 16 bytes (FSX_E_UNSUPPORTED otherwise); a shared cache
 *                  (FSX_CACHE_SHARED) is refused with FSX_E_UNSUPPORTED
 *   policy         FSX_APPEND_RING: when a ring is full the oldest rows are overwritten (start
 *                  advances); FSX_APPEND_ERROR: FSX_E_CAPACITY if any agent would exceed
 *                  capacity, and nothing is written.
 * The row copy is enqueued on `stream` (bit-exact); len/start/pos in the descriptor are
 * updated on the host before returning (pos advances by n_rows), so later calls enqueued
 * on the same stream see the new rows. */
int fsx_cache_append_rows(fsx_cache_desc* cache, const void* k_rows, const void* v_rows, int32_t n_rows,
                          int32_t policy, void* stream);

/* The slow system's rows, quantised on the way in: rows in BF16 or F32 (rows_dtype) are stored into an
 * FP8_E4M3 cache as code = round-to-nearest-even(clamp(x / scale, -448, 448)) with the cache's existing
 * per-(agent, layer, head) k_scale / v_scale (Sec. 3.3 append; the fp8 cache of the long-context workload).
 * Layout, policy, ring update and errors as fsx_cache_append_rows; FSX_E_INVALID if the cache is not FP8 or has
 * no scales.  head_dim must be a multiple of 16. */
int fsx_cache_append_rows_quantize(fsx_cache_desc* cache, const void* k_rows, const void* v_rows, int32_t rows_dtype,
                                   int32_t n_rows, int32_t policy, void* stream);

/* ---- The asynchronous deployment loop (Sec. 3.3, "Asynchronous Deployment"; Fig. 1) ----
 * The expert runs every tick on `expert_stream`; the slow system's rows are appended on `append_stream` (a
 * different stream of the same priority).  The loop keeps two copies of the ring state: ticks read the front
 * copy, appends advance the back copy.  An append is handed to the ticks (front = back, the tick's stream waiting
 * on the append's event) at the first tick after it has completed, and at the latest on the K-1-th tick after it
 * was submitted, so a tick never lags the newest submitted rows by more than K-1 ticks.  An append that overwrites
 * rows the ticks can see (ring full) first waits for the ticks already enqueued and is handed over at the next
 * tick.  The cache descriptor's device buffers must outlive the loop; its host arrays are copied at create. */
typedef struct fsx_loop fsx_loop;
typedef struct {
  int64_t tick;        /* index of this tick */
  int32_t published;   /* 1 if this tick is the first to see the rows of earlier appends */
  int32_t staleness;   /* ticks (this one included) that ran without the newest submitted rows; 0 = up to date */
  int64_t start[FSX_MAX_BATCH], len[FSX_MAX_BATCH], pos[FSX_MAX_BATCH];  /* the ring state this tick read */
} fsx_loop_tick_info;

/* append_every = K >= 1 (the paper: 4); policy FSX_APPEND_RING or FSX_APPEND_ERROR. */
int fsx_loop_create(fsx_expert* ex, const fsx_cache_desc* cache, int32_t append_every, int32_t policy,
                    void* expert_stream, void* append_stream, fsx_loop** out);
/* One control tick (arguments as fsx_expert_forward); info (nullable, HOST) receives the ring state it read. */
int fsx_loop_tick(fsx_loop* lp, const void* tokens, int32_t batch, int32_t n_frame_tokens, float* waypoints,
                  float* hidden, fsx_loop_tick_info* info);
/* Submit n_rows new rows per (agent, layer) (layout as fsx_cache_append_rows); rows_dtype equal to the cache's
 * dtype copies them, BF16 / F32 rows into an FP8 cache are quantised.  The row buffers are read on the append
 * stream: keep them unchanged until a later tick reports them published or fsx_loop_sync returns. */
int fsx_loop_append(fsx_loop* lp, const void* k_rows, const void* v_rows, int32_t rows_dtype, int32_t n_rows);
/* Wait for both streams; cache_out (nullable) receives the newest ring state (start/len/pos). */
int fsx_loop_sync(fsx_loop* lp, fsx_cache_desc* cache_out);
/* Wait for the loop's last tick and append, then free it (the expert and the cache stay the caller's). */
void fsx_loop_destroy(fsx_loop* lp);
/* Message of the calling thread's last failed loop call. */
const char* fsx_loop_last_error(void);

/* ---- The slow system's producer of the appended rows: the backbone's incremental forward (Sec. 3.3) ----
 * Every K ticks the current frame's tokens go through the frozen backbone (LLaMA-7B: 32 layers, width 4096, 32
 * heads x 128, SwiGLU 11008) as an incremental forward over its cache: at every layer each new token attends to
 * the cached rows and to the new tokens up to itself, and its rotated key and value become the layer's appended
 * row.  The cost does not depend on the history length beyond the attention over the cached rows. */
typedef struct fsx_backbone fsx_backbone;
typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, d_ffn;  /* head_dim 128; d_model and d_ffn multiples of 32 */
  int32_t max_new_rows;  /* tokens appended per call and agent (4 per frame in the paper), 1..64 */
  int32_t max_batch;     /* agents per call, 1..64 */
  int32_t dtype;         /* FSX_BF16 */
  float rope_base;       /* rotary base of the backbone (LLaMA: 10000) */
  float rms_eps;
} fsx_backbone_cfg;

/* Pack the backbone's layers (fsx_layer_weights as for the expert: wq, wk, wv [H*Dh][d], wo [d][H*Dh], w_gate,
 * w_up [d_ffn][d], w_down [d][d_ffn], norm gains [d]; DEVICE pointers, bf16) into library-owned memory.
 * Synchronises `stream`; the caller may free its buffers afterwards. */
int fsx_backbone_create(const fsx_backbone_cfg* cfg, const fsx_layer_weights* layers, void* stream,
                        fsx_backbone** out);
/* Append n_rows new tokens per agent to every layer of the cache through the incremental forward.
 *   cache   geometry equal to the backbone's (n_layers, H, Dh); BF16 (rows stored as computed) or FP8_E4M3
 *           (rows encoded with the cache's existing scales); batch must equal cache->batch; not shared
 *   tokens  DEVICE [batch][n_rows][d] bf16 embeddings of the new tokens, at positions pos[b] .. pos[b]+n_rows-1
 *   hidden  DEVICE [n_layers][batch][n_rows][d] fp32 output of every layer, or NULL
 *   policy  FSX_APPEND_RING / FSX_APPEND_ERROR as fsx_cache_append_rows; the new tokens attend to every row the
 *           ring held before the call, also to rows the append then overwrites
 * The ring state (start, len, pos) is updated on the host before returning, as fsx_cache_append_rows does. */
int fsx_backbone_append(fsx_backbone* bb, fsx_cache_desc* cache, const void* tokens, int32_t batch, int32_t n_rows,
                        float* hidden, int32_t policy, void* stream);
/* Bytes of the packed weight matrices (streamed once per call) and of the workspace. */
int fsx_backbone_info(const fsx_backbone* bb, int64_t* weight_bytes, int64_t* workspace_bytes);
/* Wait for the handle's last call, then free it. */
void fsx_backbone_destroy(fsx_backbone* bb);

/* Synchronise `stream` and report whether the ticks enqueued on this handle completed: FSX_OK, or
 * FSX_E_HIP if a tick kernel gave up on a wait (its waypoints were then written as NaN).  The
 * failure is reported once per failed tick and cleared by reporting it. */
int fsx_expert_status(fsx_expert* ex, void* stream);

/* Phase timestamps of the last tick of a handle created with FSX_FLAG_TRACE.  Synchronises `stream`,
 * then copies n_wg x n_ev values into host_out (capacity `cap` values): for workgroup w, event e
 * (0 start, 1 after the embedding, 2 + 16*l + p after phase p of layer l with p = 0 q/k/v projection,
 * 1 attention, 2 output projection, 3 gate/up, 4 down, 2 + 16*l + 5 + k sub-phase mark k; 2 + 16*n_layers
 * at the end) is the GPU real-time counter (100 MHz).  Sub-phase marks are written only by workgroups
 * that reach them and keep older values otherwise.  FSX_E_UNSUPPORTED without the flag, FSX_E_CAPACITY
 * if cap is short. */
int fsx_expert_trace(fsx_expert* ex, uint64_t* host_out, int64_t cap, int32_t* n_wg, int32_t* n_ev, void* stream);

/* Wait for the handle's last enqueued tick (not for other work on the device), then free the packed weights
 * and the workspace.  NULL is a no-op. */
void fsx_expert_destroy(fsx_expert* ex);

/* Message of the calling thread's last failed call ("" if none). */
const char* fsx_last_error(void);

/* Introspection of a handle (any pointer may be NULL):
 *   path          0 = fused bf16 path (one persistent launch per tick, or one launch per phase with
 *                 FSX_FLAG_MULTI_LAUNCH), 1 = simple per-op kernels
 *   weight_bytes  bytes of the packed weight matrices the tick streams (excludes fp32 norm gains)
 *   workspace_bytes device workspace owned by the handle */
int fsx_expert_info(const fsx_expert* ex, int32_t* path, int64_t* weight_bytes, int64_t* workspace_bytes);

/* Library version, "major.minor.patch". */
const char* fsx_version(void);

/* Measurement helper, not part of the tick: enqueue one read-only pass over `bytes` of device memory, so the
 * caller can time (with events on `stream`) the HBM read bandwidth this device reaches with a plain streaming
 * kernel -- the ceiling next to the published peak that the tick's bandwidth is quoted against.
 *   buf    DEVICE, 16-byte aligned; bytes a positive multiple of 16 (FSX_E_INVALID otherwise)
 *   mode   0: 16-byte register loads; 1: 16-byte direct loads into LDS (the attention's access)
 *   sink   DEVICE [1024] uint32 words the kernel folds a checksum into (contents are meaningless) */
int fsx_probe_hbm_read(const void* buf, int64_t bytes, int32_t mode, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FSX_H */
