// C ABI of the expert tick: validation, weight packing, workspace, split planning and the per-tick
// launch sequence.  See include/fsx.h for the contract of every entry point.

#include <algorithm>
#include <cstdio>
#include <mutex>
#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"

using namespace fsx;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIP_TRY(expr)                                                                          \
  do {                                                                                         \
    hipError_t e_ = (expr);                                                                    \
    if (e_ != hipSuccess) return fail(FSX_E_HIP, std::string(#expr ": ") + hipGetErrorString(e_)); \
  } while (0)

int esize(int dtype) { return dtype == FSX_F32 ? 4 : (dtype == FSX_BF16 ? 2 : 1); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int KSPLIT_MAX = 8;  // split factor bound of the per-phase path's split-K projections

}  // namespace

struct fsx_expert {
  fsx_expert_cfg cfg{};
  int path = 0;  // 0 fused bf16 path, 1 per-op path
  int device = 0;
  int A = 0, S_max = 0, M_max = 0, items_max = 0;
  void* wbuf = nullptr;    // packed (fused) or copied (per-op) weight matrices
  float* fbuf = nullptr;   // norm gains: [n_layers][2][d] then final [d]
  void* head_w = nullptr;  // [n_out][d] (mean-pool head) or W1 [hidden][d], then W2 [2][hidden] (query head), cfg.dtype
  float* head_b = nullptr; // query head: b1 [hidden], then b2 [2]
  QueryHead qhead{};
  void* wsbuf = nullptr;   // workspace
  int64_t weight_bytes = 0, ws_bytes = 0;
  std::vector<FastWeights> fw;
  std::vector<GenericWeights> gw;
  Workspace ws{};
  GenericWorkspace gws{};
  const float* final_norm = nullptr;
  // persistent tick kernel
  bool tick = false;
  int cu_count = 0, nx = 0;
  TickArgs ta{};            // workspace pointers; per-forward fields are filled in forward
  uint64_t* trace = nullptr;
  uint64_t epoch = 0;
  uint64_t status_seen = 0;
  hipEvent_t done = nullptr;  // recorded after every tick enqueued on the handle (destroy waits for it)
  bool backbone = false;      // the backbone's layers (fsx_backbone_*), not an expert
  int wg_per_xcd_max = 0;     // most workgroups the create-time probe placed on one XCD
};

static void free_expert(fsx_expert* ex) {
  if (!ex) return;
  if (ex->wbuf) (void)hipFree(ex->wbuf);
  if (ex->fbuf) (void)hipFree(ex->fbuf);
  if (ex->head_w) (void)hipFree(ex->head_w);
  if (ex->head_b) (void)hipFree(ex->head_b);
  if (ex->wsbuf) (void)hipFree(ex->wsbuf);
  if (ex->trace) (void)hipFree(ex->trace);
  if (ex->done) (void)hipEventDestroy(ex->done);
  delete ex;
}

static int validate_cfg(const fsx_expert_cfg* c) {
  if (!c) return fail(FSX_E_INVALID, "cfg is NULL");
  if (c->n_layers <= 0 || c->d_model <= 0 || c->n_heads <= 0 || c->head_dim <= 0 || c->d_ffn <= 0)
    return fail(FSX_E_INVALID, "n_layers, d_model, n_heads, head_dim and d_ffn must be positive");
  if (c->head_dim % 2) return fail(FSX_E_INVALID, "head_dim must be even (rotary pairs)");
  if (c->n_expert_tokens <= 0 || c->n_out <= 0) return fail(FSX_E_INVALID, "n_expert_tokens and n_out must be positive");
  if (c->max_batch <= 0 || c->max_batch > FSX_MAX_BATCH) return fail(FSX_E_INVALID, "max_batch must be in 1..64");
  if (c->max_frame_tokens < 0) return fail(FSX_E_INVALID, "max_frame_tokens must be >= 0");
  if (c->dtype != FSX_F32 && c->dtype != FSX_BF16) return fail(FSX_E_UNSUPPORTED, "weights must be F32 or BF16");
  if (!(c->rms_eps >= 0.f) || !(c->rope_base >= 0.f)) return fail(FSX_E_INVALID, "rms_eps and rope_base must be >= 0");
  if ((int64_t)c->n_heads * c->head_dim > (1 << 20) || c->d_model > (1 << 16) || c->d_ffn > (1 << 18))
    return fail(FSX_E_UNSUPPORTED, "sizes beyond the supported range");
  if (c->head_kind != FSX_HEAD_MEAN_LINEAR && c->head_kind != FSX_HEAD_QUERY_MLP)
    return fail(FSX_E_INVALID, "head_kind must be FSX_HEAD_MEAN_LINEAR or FSX_HEAD_QUERY_MLP");
  if (c->head_kind == FSX_HEAD_QUERY_MLP) {
    if (c->n_out % 2 || c->n_out / 2 > c->n_expert_tokens || c->n_out / 2 > QH_MAX_QUERIES)
      return fail(FSX_E_INVALID, "the query head needs an even n_out with n_out / 2 <= min(n_expert_tokens, 8)");
    if (c->head_hidden < 1 || c->head_hidden > 2048) return fail(FSX_E_INVALID, "head_hidden must be in 1..2048");
    if ((int64_t)(c->n_out / 2) * (c->d_model + c->head_hidden) * 4 > 64 * 1024)
      return fail(FSX_E_UNSUPPORTED, "query head rows and hidden activations beyond 64 KiB of LDS");
  }
  return FSX_OK;
}

// backbone: the layers only (no final norm, no head), run as one launch per phase with causal own rows (the
// backbone's incremental forward, fsx_backbone_*).
static int create_impl(const fsx_expert_cfg* cfg, const fsx_layer_weights* layers, const float* final_norm,
                       const fsx_head_weights* head, void* stream, fsx_expert** out, bool backbone) {
  if (!out) return fail(FSX_E_INVALID, "out is NULL");
  *out = nullptr;
  int rc = validate_cfg(cfg);
  if (rc) return rc;
  if (!backbone && (!layers || !final_norm || !head || !head->w))
    return fail(FSX_E_INVALID, "layers, final_norm and head->w must be non-NULL");
  if (backbone && !layers) return fail(FSX_E_INVALID, "layers must be non-NULL");
  if (!backbone && cfg->head_kind == FSX_HEAD_QUERY_MLP && (!head->b || !head->w2 || !head->b2))
    return fail(FSX_E_INVALID, "the query head needs w, b, w2 and b2");
  const fsx_expert_cfg& c = *cfg;
  for (int l = 0; l < c.n_layers; ++l) {
    const fsx_layer_weights& w = layers[l];
    if (!w.wq || !w.wk || !w.wv || !w.wo || !w.w_gate || !w.w_up || !w.w_down || !w.attn_norm || !w.ffn_norm)
      return fail(FSX_E_INVALID, "layer " + std::to_string(l) + " has a NULL pointer");
  }
  hipStream_t s = (hipStream_t)stream;
  fsx_expert* ex = new fsx_expert();
  ex->cfg = c;
  if (hipGetDevice(&ex->device) != hipSuccess) {
    delete ex;
    return fail(FSX_E_HIP, "hipGetDevice failed");
  }
  const int d = c.d_model, F = c.d_ffn, H = c.n_heads, Dh = c.head_dim;
  const int A = H * Dh;
  ex->A = A;
  ex->S_max = c.n_expert_tokens + c.max_frame_tokens;
  ex->M_max = c.max_batch * ex->S_max;
  const bool fused_ok = c.dtype == FSX_BF16 && Dh == 128 && d % 32 == 0 && F % 32 == 0;
  ex->path = (fused_ok && !(c.flags & FSX_FLAG_GENERIC)) ? 0 : 1;
  ex->backbone = backbone;
  if (backbone) {
    if (ex->path != 0) {
      delete ex;
      return fail(FSX_E_UNSUPPORTED, "the backbone runs bf16 weights with head_dim 128 and d, d_ffn multiples of 32");
    }
    ex->cfg.flags |= FSX_FLAG_MULTI_LAUNCH;
  }
  const int es = esize(c.dtype);
  const int64_t per_layer = (int64_t)4 * A * d + (int64_t)3 * F * d;  // elements
  const bool qh = c.head_kind == FSX_HEAD_QUERY_MLP;
  const int64_t head_elems =
      backbone ? 0 : (qh ? (int64_t)c.head_hidden * d + 2 * (int64_t)c.head_hidden : (int64_t)c.n_out * d);
  ex->weight_bytes = (per_layer * c.n_layers + head_elems) * es;

  int last = FSX_OK;
  auto cleanup = [&](int code) {
    free_expert(ex);
    return last != FSX_OK ? last : code;
  };
  auto ok = [&](hipError_t e, const char* what) -> bool {
    if (e != hipSuccess) {
      last = e == hipErrorOutOfMemory ? FSX_E_OOM : FSX_E_HIP;
      fail(last, std::string(what) + ": " + hipGetErrorString(e));
      return false;
    }
    return true;
  };

  if (!ok(hipMalloc(&ex->wbuf, (size_t)(per_layer * c.n_layers * es)), "hipMalloc(weights)")) return cleanup(FSX_E_OOM);
  if (!ok(hipMalloc((void**)&ex->fbuf, sizeof(float) * ((size_t)2 * c.n_layers * d + d)), "hipMalloc(norms)"))
    return cleanup(FSX_E_OOM);
  if (!backbone && !ok(hipMalloc(&ex->head_w, (size_t)head_elems * es), "hipMalloc(head)")) return cleanup(FSX_E_OOM);
  if (qh && !ok(hipMalloc((void**)&ex->head_b, sizeof(float) * ((size_t)c.head_hidden + 2)), "hipMalloc(head bias)"))
    return cleanup(FSX_E_OOM);

  // norm gains and head
  for (int l = 0; l < c.n_layers; ++l) {
    if (!ok(hipMemcpyAsync(ex->fbuf + (size_t)(2 * l) * d, layers[l].attn_norm, sizeof(float) * d,
                           hipMemcpyDeviceToDevice, s), "copy attn_norm") ||
        !ok(hipMemcpyAsync(ex->fbuf + (size_t)(2 * l + 1) * d, layers[l].ffn_norm, sizeof(float) * d,
                           hipMemcpyDeviceToDevice, s), "copy ffn_norm"))
      return cleanup(FSX_E_HIP);
  }
  ex->final_norm = ex->fbuf + (size_t)2 * c.n_layers * d;
  if (backbone) {
    // no final norm and no head: the incremental forward's product is the appended rows (and hidden states)
  } else if (!ok(hipMemcpyAsync((void*)ex->final_norm, final_norm, sizeof(float) * d, hipMemcpyDeviceToDevice, s),
          "copy final_norm") ||
      !ok(hipMemcpyAsync(ex->head_w, head->w, (size_t)(qh ? (int64_t)c.head_hidden * d : (int64_t)c.n_out * d) * es,
                         hipMemcpyDeviceToDevice, s), "copy head"))
    return cleanup(FSX_E_HIP);
  if (qh && !backbone) {
    char* w2 = (char*)ex->head_w + (size_t)c.head_hidden * d * es;
    if (!ok(hipMemcpyAsync(w2, head->w2, (size_t)2 * c.head_hidden * es, hipMemcpyDeviceToDevice, s), "copy head w2") ||
        !ok(hipMemcpyAsync(ex->head_b, head->b, sizeof(float) * c.head_hidden, hipMemcpyDeviceToDevice, s), "copy head b") ||
        !ok(hipMemcpyAsync(ex->head_b + c.head_hidden, head->b2, sizeof(float) * 2, hipMemcpyDeviceToDevice, s),
            "copy head b2"))
      return cleanup(FSX_E_HIP);
    ex->qhead.w1 = ex->head_w;
    ex->qhead.b1 = ex->head_b;
    ex->qhead.w2 = w2;
    ex->qhead.b2 = ex->head_b + c.head_hidden;
    ex->qhead.hidden = c.head_hidden;
  }
  ex->qhead.wdtype = c.dtype;

  char* wp = (char*)ex->wbuf;
  if (ex->path == 0) {
    for (int l = 0; l < c.n_layers; ++l) {
      const fsx_layer_weights& w = layers[l];
      const void* ptrs[7] = {w.wq, w.wk, w.wv, w.wo, w.w_gate, w.w_up, w.w_down};
      for (const void* p : ptrs)
        if (!aligned16(p)) {
          fail(FSX_E_INVALID, "bf16 weight pointers must be 16-byte aligned");
          return cleanup(FSX_E_INVALID);
        }
      FastWeights f{};
      const size_t sq = (size_t)A * d * 2;  // bytes of one [A][d] bf16 matrix
      f.wqkv = (const uint4*)wp;
      // q/k/v and gate/up read RMSNorm outputs: their gains are folded into the packed weights
      bool good =
          ok(launch_pack((const uint16_t*)w.wq, nullptr, A, d, PACK_ROPE_PAIRS, Dh, w.attn_norm, wp, s), "pack wq") &&
          ok(launch_pack((const uint16_t*)w.wk, nullptr, A, d, PACK_ROPE_PAIRS, Dh, w.attn_norm, wp + sq, s), "pack wk") &&
          ok(launch_pack((const uint16_t*)w.wv, nullptr, A, d, PACK_PLAIN, 0, w.attn_norm, wp + 2 * sq, s), "pack wv");
      wp += 3 * sq;
      f.wo = (const uint4*)wp;
      good = good && ok(launch_pack((const uint16_t*)w.wo, nullptr, d, A, PACK_PLAIN, 0, nullptr, wp, s), "pack wo");
      wp += sq;
      f.wgu = (const uint4*)wp;
      good = good && ok(launch_pack((const uint16_t*)w.w_gate, (const uint16_t*)w.w_up, 2 * F, d, PACK_SWIGLU_PAIRS, 0,
                                    w.ffn_norm, wp, s), "pack gate/up");
      wp += (size_t)2 * F * d * 2;
      f.wd = (const uint4*)wp;
      good = good && ok(launch_pack((const uint16_t*)w.w_down, nullptr, d, F, PACK_PLAIN, 0, nullptr, wp, s), "pack down");
      wp += (size_t)F * d * 2;
      if (!good) return cleanup(FSX_E_HIP);
      f.attn_norm = ex->fbuf + (size_t)(2 * l) * d;
      f.ffn_norm = ex->fbuf + (size_t)(2 * l + 1) * d;
      ex->fw.push_back(f);
    }
  } else {
    for (int l = 0; l < c.n_layers; ++l) {
      const fsx_layer_weights& w = layers[l];
      GenericWeights g{};
      const size_t n_ad = (size_t)A * d * es, n_fd = (size_t)F * d * es;
      const void* src[7] = {w.wq, w.wk, w.wv, w.wo, w.w_gate, w.w_up, w.w_down};
      const size_t sz[7] = {n_ad, n_ad, n_ad, n_ad, n_fd, n_fd, n_fd};
      const void** dst[7] = {&g.wq, &g.wk, &g.wv, &g.wo, &g.wg, &g.wu, &g.wd};
      for (int i = 0; i < 7; ++i) {
        if (!ok(hipMemcpyAsync(wp, src[i], sz[i], hipMemcpyDeviceToDevice, s), "copy weights")) return cleanup(FSX_E_HIP);
        *dst[i] = wp;
        wp += sz[i];
      }
      g.attn_norm = ex->fbuf + (size_t)(2 * l) * d;
      g.ffn_norm = ex->fbuf + (size_t)(2 * l + 1) * d;
      ex->gw.push_back(g);
    }
  }

  // workspace
  const int M = ex->M_max;
  const int n_tt_max = (ex->S_max + 15) / 16;
  {
    hipDeviceProp_t prop;
    if (!ok(hipGetDeviceProperties(&prop, ex->device), "hipGetDeviceProperties")) return cleanup(FSX_E_HIP);
    ex->cu_count = prop.multiProcessorCount;
  }
  // partial attention states: per-phase chunks, or the tick kernel's slots (NXR XCDs x (4 per agent + one per
  // workgroup)) per query tile
  ex->items_max =
      std::max({16384, 2 * c.max_batch * H * n_tt_max + 64, NXR * (4 * c.max_batch + ex->cu_count) * n_tt_max});
  std::vector<std::pair<void**, size_t>> parts;
  if (ex->path == 0) {
    parts = {{(void**)&ex->ws.h, (size_t)M * d * 4},
             {(void**)&ex->ws.xb, (size_t)M * d * 2},
             {(void**)&ex->ws.q, (size_t)M * A * 4},
             {(void**)&ex->ws.kself, (size_t)M * A * 2},
             {(void**)&ex->ws.vself, (size_t)M * A * 2},
             {(void**)&ex->ws.attn, (size_t)M * A * 2},
             {(void**)&ex->ws.z, (size_t)M * F * 2},
             {(void**)&ex->ws.part, (size_t)KSPLIT_MAX * M * d * 4},  // split factors are <= KSPLIT_MAX
             {(void**)&ex->ws.att_o, (size_t)ex->items_max * 16 * Dh * 4},
             {(void**)&ex->ws.att_ml, (size_t)ex->items_max * 32 * 4},
             {(void**)&ex->ws.rope, (size_t)M * Dh * 4},
             {(void**)&ex->ws.ss, (size_t)M * (d / 512 + 1) * 4},
             {(void**)&ex->ws.rs, (size_t)M * 4},
             {(void**)&ex->ws.rcnt, (size_t)M * 4}};
  } else {
    parts = {{(void**)&ex->gws.h, (size_t)M * d * 4},   {(void**)&ex->gws.x, (size_t)M * d * 4},
             {(void**)&ex->gws.q, (size_t)M * A * 4},   {(void**)&ex->gws.k, (size_t)M * A * 4},
             {(void**)&ex->gws.v, (size_t)M * A * 4},   {(void**)&ex->gws.attn, (size_t)M * A * 4},
             {(void**)&ex->gws.g, (size_t)M * F * 4},   {(void**)&ex->gws.u, (size_t)M * F * 4},
             {(void**)&ex->gws.rope, (size_t)M * Dh * 4}};
  }
  const int nflag_attn = c.max_batch * H;
  if (ex->path == 0 && !(ex->cfg.flags & FSX_FLAG_MULTI_LAUNCH)) {
    // The tick kernel splits heads and FFN columns over the XCDs; find how many there are and check that
    // every XCD's share fits the kernel (at most 4 heads of width 128 and 512 FFN columns per XCD).
    int nx = 0;
    if (ex->cu_count <= 512) {
      uint32_t* dev_ids = nullptr;
      std::vector<uint32_t> ids(ex->cu_count);
      if (!ok(hipMalloc((void**)&dev_ids, sizeof(uint32_t) * ex->cu_count), "hipMalloc(xcd probe)")) return cleanup(FSX_E_OOM);
      const bool good = ok(probe_xcds(dev_ids, ex->cu_count, s), "probe_xcds") &&
                        ok(hipMemcpyAsync(ids.data(), dev_ids, sizeof(uint32_t) * ex->cu_count, hipMemcpyDeviceToHost, s),
                           "copy xcd probe") &&
                        ok(hipStreamSynchronize(s), "hipStreamSynchronize(xcd probe)");
      (void)hipFree(dev_ids);
      if (!good) return cleanup(FSX_E_HIP);
      int cnt[16] = {0};
      for (uint32_t id : ids) ++cnt[id & 15];
      for (int x = 0; x < 16; ++x) {
        nx += cnt[x] > 0;
        ex->wg_per_xcd_max = std::max(ex->wg_per_xcd_max, cnt[x]);
      }
    }
    ex->nx = nx;
    const int nh_max = nx > 0 ? (H + nx - 1) / nx : 1 << 30;
    const int fr_max = nx > 0 ? 32 * ((F / 32 + nx - 1) / nx) : 1 << 30;
    ex->tick = nx > 0 && nx <= NXR && ex->cu_count <= XFLAGS && d <= 512 && d % 32 == 0 && F % 32 == 0 && nh_max <= 4 && fr_max <= 512 &&
               c.n_expert_tokens <= 64;
  }
  if (ex->tick) {
    TickArgs& t = ex->ta;
    const size_t dt = (size_t)d / 16;
    const size_t n_tt_max = ((size_t)ex->S_max + 15) / 16;
    const size_t Mp = ((size_t)M + 7) / 8 * 8, Ms = ((size_t)M + 31) / 32 * 32;
    auto r256 = [](size_t b) { return (b + 255) & ~(size_t)255; };
    const size_t rep_f = r256(Mp * d * 4), rep_b = r256(Mp * d * 2), rep_s = r256(dt * Ms * 4),
                 rep_r = r256((size_t)M * Dh * 4);
    t.x_stride_r = (int64_t)(rep_r / 4);
    const size_t G = (size_t)ex->cu_count;
    // data first, then everything that must start at zero (flags, stamped words, registration, status)
    std::vector<std::pair<void**, size_t>> tp = {
        {(void**)&t.hres, rep_f},
        {(void**)&t.xb_mid, rep_b},
        {(void**)&t.xb_out, rep_b},
        {(void**)&t.ssq_mid, rep_s},
        {(void**)&t.ssq_out, rep_s},
        {(void**)&t.rope, NXMAX * rep_r},
        {(void**)&t.z, Mp * F * 2},
        {(void**)&t.po, NXMAX * dt * Mp * 16 * 8},
        {(void**)&t.pd, NXMAX * dt * Mp * 16 * 8},
        {(void**)&t.reg, G * 8},
        {(void**)&t.f_rope, (size_t)NXMAX * XFLAGS * FPAD * 8},
        {(void**)&t.f_out, (size_t)XFLAGS * FPAD * 8},
        {(void**)&t.f_mid, (size_t)XFLAGS * FPAD * 8},
        {(void**)&t.f_q, (size_t)3 * A / 16 * ((M + 79) / 80) * FPAD * 8},  // per (tile, row block of 80 rows)
        {(void**)&t.f_attn, (size_t)nflag_attn * n_tt_max * FPAD * 8},
        {(void**)&t.f_rng, (size_t)ex->items_max * FPAD * 8},
        {(void**)&t.f_z, (size_t)F / 8 * ((M + 79) / 80) * FPAD * 8},
        {(void**)&t.status, 256}};
    parts.insert(parts.end(), tp.begin(), tp.end());
  }
  size_t total = 0;
  for (auto& p : parts) total += (p.second + 255) & ~(size_t)255;
  if (!ok(hipMalloc(&ex->wsbuf, total), "hipMalloc(workspace)")) return cleanup(FSX_E_OOM);
  ex->ws_bytes = (int64_t)total;
  char* q = (char*)ex->wsbuf;
  for (auto& p : parts) {
    *p.first = q;
    q += (p.second + 255) & ~(size_t)255;
  }
  // the per-row chunk counters of the wide-row reductions start at zero (each reduction leaves them at zero)
  if (ex->path == 0 && !ok(hipMemsetAsync(ex->ws.rcnt, 0, (size_t)M * 4, s), "hipMemsetAsync(row counters)"))
    return cleanup(FSX_E_HIP);
  if (ex->tick) {
    // stamped words, flags, registration and status start at zero; stamps only grow
    TickArgs& t = ex->ta;
    const size_t zbytes = (size_t)((char*)q - (char*)t.po);
    if (!ok(hipMemsetAsync(t.po, 0, zbytes, s), "hipMemsetAsync(flags)")) return cleanup(FSX_E_HIP);
    t.wbase = (const char*)ex->wbuf;
    t.final_norm = ex->final_norm;
    t.head_w = ex->head_w;
    t.head_dtype = c.dtype;
    t.qhead = ex->qhead;
    t.q = ex->ws.q;
    t.kself = ex->ws.kself;
    t.vself = ex->ws.vself;
    t.attn = ex->ws.attn;
    t.att_o = ex->ws.att_o;
    t.att_ml = ex->ws.att_ml;
    const uint64_t us = c.tick_timeout_us > 0 ? (uint64_t)c.tick_timeout_us : 2000000ull;
    t.timeout_ticks = us * 100;  // the real-time counter runs at 100 MHz
    if (c.flags & FSX_FLAG_TRACE) {
      const size_t nt = (size_t)ex->cu_count * trace_events(c.n_layers);
      if (!ok(hipMalloc((void**)&ex->trace, nt * 8), "hipMalloc(trace)") ||
          !ok(hipMemsetAsync(ex->trace, 0, nt * 8, s), "hipMemsetAsync(trace)"))
        return cleanup(FSX_E_HIP);
      t.trace = ex->trace;
    }
  }
  if (!ok(hipEventCreateWithFlags(&ex->done, hipEventDisableTiming), "hipEventCreateWithFlags")) return cleanup(FSX_E_HIP);
  if (!ok(hipStreamSynchronize(s), "hipStreamSynchronize(create)")) return cleanup(FSX_E_HIP);
  *out = ex;
  g_err.clear();
  return FSX_OK;
}

extern "C" int fsx_expert_create(const fsx_expert_cfg* cfg, const fsx_layer_weights* layers, const float* final_norm,
                                 const fsx_head_weights* head, void* stream, fsx_expert** out) {
  return create_impl(cfg, layers, final_norm, head, stream, out, false);
}

static int validate_cache(const fsx_expert* ex, const fsx_cache_desc* c, int batch) {
  if (!c) return fail(FSX_E_INVALID, "cache is NULL");
  if (c->dtype != FSX_F32 && c->dtype != FSX_BF16 && c->dtype != FSX_FP8_E4M3)
    return fail(FSX_E_INVALID, "cache dtype must be F32, BF16 or FP8_E4M3");
  if (ex && (c->n_layers != ex->cfg.n_layers || c->n_heads != ex->cfg.n_heads || c->head_dim != ex->cfg.head_dim))
    return fail(FSX_E_INVALID, "cache geometry (n_layers, n_heads, head_dim) differs from the expert's");
  if (c->layout & ~(FSX_CACHE_TOKEN_MAJOR | FSX_CACHE_SHARED))
    return fail(FSX_E_INVALID, "cache layout must be FSX_CACHE_HEAD_MAJOR or FSX_CACHE_TOKEN_MAJOR, optionally with "
                               "FSX_CACHE_SHARED");
  if (c->batch <= 0 || c->batch > FSX_MAX_BATCH) return fail(FSX_E_INVALID, "cache batch must be in 1..64");
  if (batch > c->batch) return fail(FSX_E_INVALID, "batch exceeds the cache descriptor's batch");
  if (c->capacity < 0 || c->capacity > (int64_t)INT32_MAX) return fail(FSX_E_INVALID, "capacity out of range");
  if (!c->start || !c->len || !c->pos) return fail(FSX_E_INVALID, "start, len and pos must be non-NULL host arrays");
  bool any = false;
  for (int b = 0; b < batch; ++b) {
    if (c->len[b] < 0 || c->len[b] > c->capacity)
      return fail(FSX_E_CAPACITY, "len[" + std::to_string(b) + "] outside 0..capacity");
    if (c->len[b] > 0 && (c->start[b] < 0 || c->start[b] >= c->capacity))
      return fail(FSX_E_INVALID, "start[" + std::to_string(b) + "] outside 0..capacity-1");
    if (c->pos[b] < 0 || c->pos[b] > ((int64_t)1 << 40)) return fail(FSX_E_INVALID, "pos out of range");
    any = any || c->len[b] > 0;
  }
  if (any && (!c->k || !c->v)) return fail(FSX_E_INVALID, "cache k/v pointers are NULL");
  if (any && c->dtype == FSX_FP8_E4M3 && (!c->k_scale || !c->v_scale))
    return fail(FSX_E_INVALID, "fp8 cache needs k_scale and v_scale");
  if (any && (!aligned16(c->k) || !aligned16(c->v))) return fail(FSX_E_INVALID, "cache k/v must be 16-byte aligned");
  return FSX_OK;
}

// ------------------------------------------------------------------------------------------------------------
// The entry point that allocates nothing keeps the tick kernel's workspace in `scratch`, a file-scope device array
// of STATIC_SCRATCH_BYTES.  In host code `scratch` names a host-side stand-in, never a device address: the device
// address is looked up once per device (hipGetSymbolAddress, with that device current) and only that pointer is
// used.  Every call on a device shares its array; a call clears the part that must start at zero (flags, stamped
// partial words, registration and status words) with a fill kernel on its stream, so calls are independent of the
// previous contents, but calls that overlap on one device (two streams, two threads) race on the array.
constexpr size_t STATIC_SCRATCH_BYTES = (size_t)48 << 20;
constexpr int STATIC_MAX_DEVICES = 64;
static __device__ __align__(256) uint8_t scratch[STATIC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_dev[STATIC_MAX_DEVICES] = {};

// Device address of `scratch` on device dev (the current device), looked up on the first call for that device.
int scratch_of(int dev, void** out) {
  if (dev < 0 || dev >= STATIC_MAX_DEVICES) return fail(FSX_E_UNSUPPORTED, "device index beyond the static workspace table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(FSX_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return FSX_OK;
}

// Lay the tick kernel's workspace for this call's sizes over `base` (nullptr: only measure).  Data first, then the
// part that must start at zero, from *zero_off to the returned total.
size_t static_tick_layout(const fsx_expert* ex, const TickParams& tp, char* base, TickArgs& t, size_t* zero_off) {
  const fsx_expert_cfg& c = ex->cfg;
  const size_t d = c.d_model, F = c.d_ffn, Dh = c.head_dim, A = ex->A, M = tp.M, Mp = tp.Mp, Ms = tp.Ms;
  const size_t dt = d / 16, R = ((size_t)tp.M + 79) / 80, NXS = NXR;  // per-XCD copies (rope, partials, registration): the tick path runs on <= NXR XCDs
  const size_t items = (size_t)NXR * tp.slot_x * tp.n_tt;
  auto r256 = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t rep_f = r256(Mp * d * 4), rep_b = r256(Mp * d * 2), rep_s = r256(dt * Ms * 4), rep_r = r256(M * Dh * 4);
  t.x_stride_r = (int64_t)(rep_r / 4);
  void* dummy;
  const std::pair<void**, size_t> parts[] = {
      {(void**)&t.q, M * A * 4},  {(void**)&t.kself, M * A * 2}, {(void**)&t.vself, M * A * 2},
      {(void**)&t.attn, M * A * 2}, {(void**)&t.att_o, items * 16 * Dh * 4}, {(void**)&t.att_ml, items * 32 * 4},
      {(void**)&t.hres, rep_f}, {(void**)&t.xb_mid, rep_b}, {(void**)&t.xb_out, rep_b},
      {(void**)&t.ssq_mid, rep_s}, {(void**)&t.ssq_out, rep_s}, {(void**)&t.rope, NXS * rep_r},
      {(void**)&t.z, Mp * F * 2},
      {&dummy, 0},  // start of the part that must start at zero
      {(void**)&t.po, NXS * dt * Mp * 16 * 8}, {(void**)&t.pd, NXS * dt * Mp * 16 * 8},
      {(void**)&t.reg, (size_t)ex->cu_count * 8}, {(void**)&t.f_rope, NXS * XFLAGS * FPAD * 8},
      {(void**)&t.f_out, XFLAGS * FPAD * 8}, {(void**)&t.f_mid, XFLAGS * FPAD * 8},
      {(void**)&t.f_q, 3 * A / 16 * R * FPAD * 8}, {(void**)&t.f_attn, (size_t)tp.B * c.n_heads * tp.n_tt * FPAD * 8},
      {(void**)&t.f_rng, items * FPAD * 8}, {(void**)&t.f_z, F / 8 * R * FPAD * 8}, {(void**)&t.status, 256}};
  size_t off = 0;
  for (const auto& p : parts) {
    if (p.first == &dummy) {
      *zero_off = off;
      continue;
    }
    if (base) *p.first = base + off;
    off += r256(p.second);
  }
  return off;
}
}  // namespace

static int forward_impl(fsx_expert* ex, const fsx_cache_desc* cache, const void* tokens, int32_t batch,
                        int32_t n_frame_tokens, float* waypoints, float* hidden, void* stream, bool use_static) {
  if (!ex) return fail(FSX_E_INVALID, "expert handle is NULL");
  if (!tokens || !waypoints) return fail(FSX_E_INVALID, "tokens and waypoints must be non-NULL");
  const fsx_expert_cfg& c = ex->cfg;
  if (batch <= 0) return fail(FSX_E_INVALID, "batch must be positive");
  if (batch > c.max_batch) return fail(FSX_E_CAPACITY, "batch exceeds max_batch");
  if (n_frame_tokens < 0 || n_frame_tokens > c.max_frame_tokens)
    return fail(FSX_E_CAPACITY, "n_frame_tokens outside 0..max_frame_tokens");
  int rc = validate_cache(ex, cache, batch);
  if (rc) return rc;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != ex->device) return fail(FSX_E_INVALID, "current device differs from the one the expert was created on");
  if (ex->path == 0 && cache->dtype == FSX_F32) return fail(FSX_E_UNSUPPORTED, "the bf16 expert reads BF16 or FP8 caches");
  if (ex->path == 0 && !aligned16(tokens)) return fail(FSX_E_INVALID, "tokens must be 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;

  TickParams tp{};
  tp.B = batch;
  tp.S = c.n_expert_tokens + n_frame_tokens;
  tp.T = c.n_expert_tokens;
  tp.M = batch * tp.S;
  tp.n_tt = (tp.S + 15) / 16;
  int64_t rows = 0;
  for (int b = 0; b < batch; ++b) {
    tp.pos[b] = cache->pos[b];
    tp.start[b] = cache->len[b] > 0 ? cache->start[b] : 0;
    tp.len[b] = (int32_t)cache->len[b];
    rows += cache->len[b];
  }
  Dims dm{};
  dm.d = c.d_model; dm.H = c.n_heads; dm.Dh = c.head_dim; dm.A = ex->A; dm.F = c.d_ffn; dm.n_layers = c.n_layers;
  dm.n_out = c.n_out; dm.eps = c.rms_eps; dm.rope_base = c.rope_base; dm.head_kind = c.head_kind;
  CacheView cv{};
  cv.k = cache->k; cv.v = cache->v; cv.k_scale = cache->k_scale; cv.v_scale = cache->v_scale;
  cv.cap = cache->capacity; cv.n_layers = cache->n_layers; cv.layer = 0; cv.dtype = cache->dtype;
  cv.H = cache->n_heads; cv.Dh = cache->head_dim;
  const bool shared = (cache->layout & FSX_CACHE_SHARED) != 0;
  cv.bs = shared ? 0 : (int64_t)cache->n_layers * cache->n_heads * cache->capacity * cache->head_dim;
  cv.sbs = shared ? 0 : cache->n_layers * cache->n_heads;
  if (cache->layout & FSX_CACHE_TOKEN_MAJOR) {
    cv.hs = cache->head_dim;
    cv.rs = (int64_t)cache->n_heads * cache->head_dim;
  } else {
    cv.hs = cache->capacity * cache->head_dim;
    cv.rs = cache->head_dim;
  }

  if (use_static && !ex->tick)
    return fail(FSX_E_UNSUPPORTED, "the allocation-free entry point runs the persistent tick kernel only (bf16 expert "
                                   "whose heads and FFN columns fit the per-XCD split, no FSX_FLAG_MULTI_LAUNCH)");
  if (ex->path == 1) {
    HIP_TRY(generic_tick(ex->gw.data(), ex->final_norm, ex->head_w, ex->qhead, c.dtype, tokens, cv, tp, dm, ex->gws,
                         waypoints, hidden, s));
    HIP_TRY(hipEventRecord(ex->done, s));
    g_err.clear();
    return FSX_OK;
  }

  // split plan: chunk rows (multiple of 32) so that the work items number about 2048
  const int target = 2048;
  const int64_t work = rows * dm.H * tp.n_tt;
  int64_t cr = (work + target - 1) / target;
  cr = std::max<int64_t>(32, ((cr + 31) / 32) * 32);
  int n_items = 0;
  for (;;) {
    int64_t slots = 0;
    for (int b = 0; b < batch; ++b) slots += (tp.len[b] + cr - 1) / cr + 1;
    const int64_t items = slots * dm.H * tp.n_tt;
    if (items <= ex->items_max) {
      n_items = (int)items;
      break;
    }
    cr *= 2;
  }
  tp.chunk_rows = (int)cr;
  tp.n_items = n_items;
  tp.chunk_prefix[0] = 0;
  for (int b = 0; b < batch; ++b) tp.chunk_prefix[b + 1] = tp.chunk_prefix[b] + (int)((tp.len[b] + cr - 1) / cr) + 1;
  if (ex->tick) {
    int per_cu = 0;
    HIP_TRY(tick_occupancy(cache->dtype == FSX_FP8_E4M3 ? 1 : 0, &per_cu));
    if (per_cu < 1) return fail(FSX_E_UNSUPPORTED, "tick kernel does not fit on a compute unit");
    const int G = ex->cu_count;
    tp.Mp = (tp.M + 7) / 8 * 8;
    tp.Ms = (tp.M + 31) / 32 * 32;
    // row blocks per residual column tile: about one piece per workgroup, pieces of at least 16 rows (the pieces
    // number at most G <= XFLAGS, the flag slots of f_out and f_mid)
    tp.rblk = std::max(1, std::min(G / (dm.d / 16), (tp.M + 15) / 16));
    // Attention work (the kernel slices it): agents longest first; per head, agent b weighs its 32-row cache
    // tiles followed by the 32-row tiles of the expert's own rows
    std::vector<int> ord(batch);
    for (int b = 0; b < batch; ++b) ord[b] = b;
    std::stable_sort(ord.begin(), ord.end(), [&](int x, int y) { return tp.len[x] > tp.len[y]; });
    tp.seg_p[0] = 0;
    for (int k = 0; k < batch; ++k) {
      const int b = ord[k];
      tp.order[k] = b;
      tp.seg_w[k] = (int)((tp.len[b] + 31) / 32) + (tp.S + 31) / 32;
      tp.seg_p[k + 1] = tp.seg_p[k] + tp.seg_w[k];
    }
    // partial-state slots per XCD: at most one per segment (<= 4 local heads per agent) plus one per slice boundary
    // (the kernel checks the bound and fails the tick if the placement breaks it)
    tp.slot_x = batch * 4 + (use_static ? ex->wg_per_xcd_max : G);
    TickArgs a = ex->ta;
    if (use_static) {
      // the workspace for this call's sizes, laid over the static array; epoch 1 on flags cleared by this call
      size_t zoff = 0;
      const size_t need = static_tick_layout(ex, tp, nullptr, a, &zoff);
      if (need > STATIC_SCRATCH_BYTES)
        return fail(FSX_E_CAPACITY, "this call needs " + std::to_string(need) + " bytes of workspace; the static array "
                                    "holds " + std::to_string(STATIC_SCRATCH_BYTES));
      void* base = nullptr;
      rc = scratch_of(dev, &base);
      if (rc) return rc;
      static_tick_layout(ex, tp, (char*)base, a, &zoff);
      HIP_TRY(launch_fill_zero((char*)base + zoff, need - zoff, s));
      a.epoch = 1;
    } else {
      if ((int64_t)NXR * tp.slot_x * tp.n_tt > ex->items_max)
        return fail(FSX_E_UNSUPPORTED, "attention partial-state slots exceed the workspace");
      a.epoch = ++ex->epoch;
    }
    a.tok_dtype = c.dtype;
    a.tokens = tokens;
    a.cv = cv;
    a.waypoints = waypoints;
    a.hidden = hidden;
    HIP_TRY(launch_tick(a, tp, dm, ex->cu_count, s));
    HIP_TRY(hipEventRecord(ex->done, s));
    g_err.clear();
    return FSX_OK;
  }
  const int wpg = n_items >= 1024 ? 4 : 1;
  auto kspl = [](int KB) { return KB % 8 == 0 ? 8 : (KB % 4 == 0 ? 4 : (KB % 2 == 0 ? 2 : 1)); };
  const int ks_o = kspl(dm.A / 32), ks_d = kspl(dm.F / 32);

  HIP_TRY(launch_embed(tokens, c.dtype, ex->fw[0].attn_norm, tp, dm, ex->ws, s));
  for (int l = 0; l < c.n_layers; ++l) {
    const FastWeights& w = ex->fw[l];
    cv.layer = l;
    HIP_TRY(launch_gemm_qkv(w, tp, dm, ex->ws, s, l > 0));
    HIP_TRY(launch_attention(cv, tp, dm, ex->ws, wpg, s));
    HIP_TRY(launch_combine(tp, dm, ex->ws, s));
    HIP_TRY(launch_gemm_o(w, tp, dm, ex->ws, ks_o, s));
    HIP_TRY(launch_reduce_norm(tp, dm, ex->ws, ks_o, w.ffn_norm, nullptr, s));
    HIP_TRY(launch_gemm_gu(w, tp, dm, ex->ws, s));
    HIP_TRY(launch_gemm_down(w, tp, dm, ex->ws, ks_d, s));
    const float* gnext = l + 1 < c.n_layers ? ex->fw[l + 1].attn_norm : ex->final_norm;
    HIP_TRY(launch_reduce_norm(tp, dm, ex->ws, ks_d, gnext, hidden ? hidden + (int64_t)l * tp.M * dm.d : nullptr, s));
  }
  if (c.head_kind == FSX_HEAD_QUERY_MLP)
    HIP_TRY(launch_query_head(ex->ws.h, tp, dm, ex->final_norm, ex->qhead, waypoints, s));
  else
    HIP_TRY(launch_head(tp, dm, ex->ws, ex->final_norm, ex->head_w, c.dtype, waypoints, s));
  HIP_TRY(hipEventRecord(ex->done, s));
  g_err.clear();
  return FSX_OK;
}

extern "C" int fsx_expert_forward(fsx_expert* ex, const fsx_cache_desc* cache, const void* tokens, int32_t batch,
                                  int32_t n_frame_tokens, float* waypoints, float* hidden, void* stream) {
  return forward_impl(ex, cache, tokens, batch, n_frame_tokens, waypoints, hidden, stream, false);
}

extern "C" int fsx_expert_forward_noalloc(fsx_expert* ex, const fsx_cache_desc* cache, const void* tokens,
                                          int32_t batch, int32_t n_frame_tokens, float* waypoints, float* hidden,
                                          void* stream) {
  return forward_impl(ex, cache, tokens, batch, n_frame_tokens, waypoints, hidden, stream, true);
}

// rows_dtype < 0: rows in the cache's dtype (bit copy); else bf16 / fp32 rows encoded into an fp8 cache.
static int append_impl(fsx_cache_desc* cache, const void* k_rows, const void* v_rows, int rows_dtype, int32_t n_rows,
                       int32_t policy, void* stream) {
  int rc = validate_cache(nullptr, cache, cache ? cache->batch : 0);
  if (rc) return rc;
  if (n_rows < 0) return fail(FSX_E_INVALID, "n_rows must be >= 0");
  if (policy != FSX_APPEND_RING && policy != FSX_APPEND_ERROR) return fail(FSX_E_INVALID, "unknown append policy");
  if (rows_dtype >= 0) {
    if (cache->dtype != FSX_FP8_E4M3) return fail(FSX_E_INVALID, "quantising append needs an FP8_E4M3 cache");
    if (rows_dtype != FSX_BF16 && rows_dtype != FSX_F32) return fail(FSX_E_INVALID, "rows must be BF16 or F32");
    if (!cache->k_scale || !cache->v_scale) return fail(FSX_E_INVALID, "fp8 cache needs k_scale and v_scale");
  }
  if (n_rows == 0) {
    g_err.clear();
    return FSX_OK;
  }
  if (!k_rows || !v_rows || !cache->k || !cache->v) return fail(FSX_E_INVALID, "row and cache pointers must be non-NULL");
  if (n_rows > cache->capacity) return fail(FSX_E_CAPACITY, "n_rows exceeds the ring capacity");
  if (cache->layout & FSX_CACHE_SHARED)
    return fail(FSX_E_UNSUPPORTED, "a shared cache is a set of views of one agent's rings; append through a "
                                   "descriptor of that agent alone");
  if (cache->n_layers <= 0 || cache->n_heads <= 0 || cache->head_dim <= 0)
    return fail(FSX_E_INVALID, "cache geometry must be positive");
  const int64_t head_row_bytes = (int64_t)cache->head_dim * esize(cache->dtype);
  if (head_row_bytes % 16) return fail(FSX_E_UNSUPPORTED, "a cache row of one head must be a multiple of 16 bytes");
  if (!aligned16(k_rows) || !aligned16(v_rows) || !aligned16(cache->k) || !aligned16(cache->v))
    return fail(FSX_E_INVALID, "row and cache buffers must be 16-byte aligned");
  const int B = cache->batch;
  if (policy == FSX_APPEND_ERROR)
    for (int b = 0; b < B; ++b)
      if (cache->len[b] + n_rows > cache->capacity)
        return fail(FSX_E_CAPACITY, "agent " + std::to_string(b) + ": ring full (policy FSX_APPEND_ERROR)");
  std::vector<int64_t> first(B);
  for (int b = 0; b < B; ++b) {
    const int64_t st = cache->len[b] > 0 ? cache->start[b] : 0;
    first[b] = (st + cache->len[b]) % cache->capacity;
  }
  if (rows_dtype >= 0)
    HIP_TRY(launch_append_quantize(*cache, k_rows, v_rows, rows_dtype, n_rows, first.data(), (hipStream_t)stream));
  else
    HIP_TRY(launch_append(*cache, k_rows, v_rows, n_rows, first.data(), (hipStream_t)stream));
  for (int b = 0; b < B; ++b) {
    const int64_t st = cache->len[b] > 0 ? cache->start[b] : first[b];
    const int64_t nl = cache->len[b] + n_rows;
    if (nl <= cache->capacity) {
      cache->start[b] = st;
      cache->len[b] = nl;
    } else {  // ring: the oldest rows were overwritten
      cache->start[b] = (st + (nl - cache->capacity)) % cache->capacity;
      cache->len[b] = cache->capacity;
    }
    cache->pos[b] += n_rows;
  }
  g_err.clear();
  return FSX_OK;
}

extern "C" int fsx_cache_append_rows(fsx_cache_desc* cache, const void* k_rows, const void* v_rows, int32_t n_rows,
                                     int32_t policy, void* stream) {
  return append_impl(cache, k_rows, v_rows, -1, n_rows, policy, stream);
}

extern "C" int fsx_cache_append_rows_quantize(fsx_cache_desc* cache, const void* k_rows, const void* v_rows,
                                              int32_t rows_dtype, int32_t n_rows, int32_t policy, void* stream) {
  if (rows_dtype < 0) return fail(FSX_E_INVALID, "rows must be BF16 or F32");
  return append_impl(cache, k_rows, v_rows, rows_dtype, n_rows, policy, stream);
}

extern "C" int fsx_expert_status(fsx_expert* ex, void* stream) {
  if (!ex) return fail(FSX_E_INVALID, "expert handle is NULL");
  HIP_TRY(hipStreamSynchronize((hipStream_t)stream));
  if (!ex->tick) {
    g_err.clear();
    return FSX_OK;
  }
  uint64_t v = 0;
  HIP_TRY(hipMemcpy(&v, ex->ta.status, sizeof(v), hipMemcpyDeviceToHost));
  if (v != ex->status_seen) {
    ex->status_seen = v;
    return fail(FSX_E_HIP, "a tick kernel timed out waiting for another workgroup (tick " + std::to_string(v - 1) +
                               "); its waypoints are NaN");
  }
  g_err.clear();
  return FSX_OK;
}

extern "C" int fsx_expert_trace(fsx_expert* ex, uint64_t* host_out, int64_t cap, int32_t* n_wg, int32_t* n_ev,
                                void* stream) {
  if (!ex || !host_out) return fail(FSX_E_INVALID, "expert handle and host_out must be non-NULL");
  if (!ex->trace) return fail(FSX_E_UNSUPPORTED, "the handle was not created with FSX_FLAG_TRACE");
  const int64_t n = (int64_t)ex->cu_count * trace_events(ex->cfg.n_layers);
  if (cap < n) return fail(FSX_E_CAPACITY, "host_out holds fewer than n_wg * n_ev values");
  HIP_TRY(hipStreamSynchronize((hipStream_t)stream));
  HIP_TRY(hipMemcpy(host_out, ex->trace, (size_t)n * 8, hipMemcpyDeviceToHost));
  if (n_wg) *n_wg = ex->cu_count;
  if (n_ev) *n_ev = trace_events(ex->cfg.n_layers);
  g_err.clear();
  return FSX_OK;
}

extern "C" void fsx_expert_destroy(fsx_expert* ex) {
  if (!ex) return;
  if (ex->done) (void)hipEventSynchronize(ex->done);  // the handle's last tick, not the whole device
  free_expert(ex);
}

extern "C" const char* fsx_last_error(void) { return g_err.c_str(); }

extern "C" int fsx_expert_info(const fsx_expert* ex, int32_t* path, int64_t* weight_bytes, int64_t* workspace_bytes) {
  if (!ex) return fail(FSX_E_INVALID, "expert handle is NULL");
  if (path) *path = ex->path;  // the tick kernel and the per-phase launches are both path 0
  if (weight_bytes) *weight_bytes = ex->weight_bytes;
  if (workspace_bytes) *workspace_bytes = ex->ws_bytes;
  return FSX_OK;
}

extern "C" const char* fsx_version(void) { return "0.2.0"; }

extern "C" int fsx_probe_hbm_read(const void* buf, int64_t bytes, int32_t mode, uint32_t* sink, void* stream) {
  if (!buf || !sink) return fail(FSX_E_INVALID, "buf and sink must be non-NULL");
  if (bytes <= 0 || bytes % 16 || !aligned16(buf)) return fail(FSX_E_INVALID, "bytes must be a positive multiple of 16 and buf 16-byte aligned");
  if (mode != 0 && mode != 1) return fail(FSX_E_INVALID, "mode must be 0 or 1");
  HIP_TRY(launch_probe_read(buf, bytes, mode, sink, (hipStream_t)stream));
  g_err.clear();
  return FSX_OK;
}

// ------------------------------------------------------------------------------------------------------------
// The backbone's incremental forward (Sec. 3.3): the slow system's producer of the appended rows.  The layers run
// as one launch per phase (split-K MFMA projections streaming the packed weights, split-K attention over the
// cached rows plus the new rows under a causal mask); after each layer's attention the new rows' rotated keys and
// values are written into that layer's ring slots.
struct fsx_backbone {
  fsx_expert* ex = nullptr;
};

extern "C" int fsx_backbone_create(const fsx_backbone_cfg* cfg, const fsx_layer_weights* layers, void* stream,
                                   fsx_backbone** out) {
  if (!out) return fail(FSX_E_INVALID, "out is NULL");
  *out = nullptr;
  if (!cfg) return fail(FSX_E_INVALID, "cfg is NULL");
  if (cfg->dtype != FSX_BF16) return fail(FSX_E_UNSUPPORTED, "the backbone runs bf16 weights");
  if (cfg->max_new_rows < 1 || cfg->max_new_rows > 64) return fail(FSX_E_INVALID, "max_new_rows must be in 1..64");
  fsx_expert_cfg c{};
  c.n_layers = cfg->n_layers; c.d_model = cfg->d_model; c.n_heads = cfg->n_heads; c.head_dim = cfg->head_dim;
  c.d_ffn = cfg->d_ffn; c.n_expert_tokens = cfg->max_new_rows; c.n_out = 2; c.max_batch = cfg->max_batch;
  c.max_frame_tokens = 0; c.dtype = cfg->dtype; c.rope_base = cfg->rope_base; c.rms_eps = cfg->rms_eps;
  c.flags = FSX_FLAG_MULTI_LAUNCH; c.head_kind = FSX_HEAD_MEAN_LINEAR;
  fsx_expert* ex = nullptr;
  const int rc = create_impl(&c, layers, nullptr, nullptr, stream, &ex, true);
  if (rc) return rc;
  fsx_backbone* bb = new fsx_backbone();
  bb->ex = ex;
  *out = bb;
  g_err.clear();
  return FSX_OK;
}

extern "C" int fsx_backbone_append(fsx_backbone* bb, fsx_cache_desc* cache, const void* tokens, int32_t batch,
                                   int32_t n_rows, float* hidden, int32_t policy, void* stream) {
  if (!bb || !bb->ex) return fail(FSX_E_INVALID, "backbone handle is NULL");
  fsx_expert* ex = bb->ex;
  const fsx_expert_cfg& c = ex->cfg;
  if (!tokens) return fail(FSX_E_INVALID, "tokens must be non-NULL");
  if (n_rows < 1 || n_rows > c.n_expert_tokens) return fail(FSX_E_CAPACITY, "n_rows outside 1..max_new_rows");
  if (policy != FSX_APPEND_RING && policy != FSX_APPEND_ERROR) return fail(FSX_E_INVALID, "unknown append policy");
  int rc = validate_cache(ex, cache, batch);
  if (rc) return rc;
  if (batch != cache->batch) return fail(FSX_E_INVALID, "the backbone appends to every agent of the descriptor: batch "
                                                        "must equal cache->batch");
  if (batch > c.max_batch) return fail(FSX_E_CAPACITY, "batch exceeds max_batch");
  if (cache->layout & FSX_CACHE_SHARED) return fail(FSX_E_UNSUPPORTED, "a shared cache cannot be appended to");
  if (cache->dtype != FSX_BF16 && cache->dtype != FSX_FP8_E4M3)
    return fail(FSX_E_UNSUPPORTED, "the backbone writes BF16 or FP8 caches");
  if (!cache->k || !cache->v) return fail(FSX_E_INVALID, "cache k/v pointers are NULL");
  if (cache->dtype == FSX_FP8_E4M3 && (!cache->k_scale || !cache->v_scale))
    return fail(FSX_E_INVALID, "fp8 cache needs k_scale and v_scale");
  if (!aligned16(tokens) || !aligned16(cache->k) || !aligned16(cache->v))
    return fail(FSX_E_INVALID, "tokens and cache buffers must be 16-byte aligned");
  if (n_rows > cache->capacity) return fail(FSX_E_CAPACITY, "n_rows exceeds the ring capacity");
  if (policy == FSX_APPEND_ERROR)
    for (int b = 0; b < batch; ++b)
      if (cache->len[b] + n_rows > cache->capacity)
        return fail(FSX_E_CAPACITY, "agent " + std::to_string(b) + ": ring full (policy FSX_APPEND_ERROR)");
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != ex->device) return fail(FSX_E_INVALID, "current device differs from the one the backbone was created on");
  hipStream_t s = (hipStream_t)stream;

  TickParams tp{};
  tp.B = batch;
  tp.S = n_rows;
  tp.T = n_rows;
  tp.M = batch * n_rows;
  tp.n_tt = (tp.S + 15) / 16;
  int64_t rows = 0;
  std::vector<int64_t> first(batch);
  for (int b = 0; b < batch; ++b) {
    tp.pos[b] = cache->pos[b];  // the new tokens sit at positions pos .. pos + n_rows - 1
    tp.start[b] = cache->len[b] > 0 ? cache->start[b] : 0;
    tp.len[b] = (int32_t)cache->len[b];
    rows += cache->len[b];
    first[b] = (tp.start[b] + cache->len[b]) % cache->capacity;
  }
  Dims dm{};
  dm.d = c.d_model; dm.H = c.n_heads; dm.Dh = c.head_dim; dm.A = ex->A; dm.F = c.d_ffn; dm.n_layers = c.n_layers;
  dm.n_out = c.n_out; dm.eps = c.rms_eps; dm.rope_base = c.rope_base; dm.head_kind = 0;
  CacheView cv{};
  cv.k = cache->k; cv.v = cache->v; cv.k_scale = cache->k_scale; cv.v_scale = cache->v_scale;
  cv.cap = cache->capacity; cv.n_layers = cache->n_layers; cv.dtype = cache->dtype;
  cv.H = cache->n_heads; cv.Dh = cache->head_dim;
  cv.bs = (int64_t)cache->n_layers * cache->n_heads * cache->capacity * cache->head_dim;
  cv.sbs = cache->n_layers * cache->n_heads;
  if (cache->layout & FSX_CACHE_TOKEN_MAJOR) {
    cv.hs = cache->head_dim;
    cv.rs = (int64_t)cache->n_heads * cache->head_dim;
  } else {
    cv.hs = cache->capacity * cache->head_dim;
    cv.rs = cache->head_dim;
  }
  // split plan of the attention over the cached rows (as the per-phase expert tick)
  const int target = 2048;
  const int64_t work = rows * dm.H * tp.n_tt;
  int64_t cr = std::max<int64_t>(32, (((work + target - 1) / target + 31) / 32) * 32);
  for (;;) {
    int64_t slots = 0;
    for (int b = 0; b < batch; ++b) slots += (tp.len[b] + cr - 1) / cr + 1;
    if (slots * dm.H * tp.n_tt <= ex->items_max) {
      tp.n_items = (int)(slots * dm.H * tp.n_tt);
      break;
    }
    cr *= 2;
  }
  tp.chunk_rows = (int)cr;
  tp.chunk_prefix[0] = 0;
  for (int b = 0; b < batch; ++b) tp.chunk_prefix[b + 1] = tp.chunk_prefix[b] + (int)((tp.len[b] + cr - 1) / cr) + 1;
  const int wpg = tp.n_items >= 1024 ? 4 : 1;
  auto kspl = [](int KB) { return KB % 8 == 0 ? 8 : (KB % 4 == 0 ? 4 : (KB % 2 == 0 ? 2 : 1)); };
  const int ks_o = kspl(dm.A / 32), ks_d = kspl(dm.F / 32);
  HIP_TRY(launch_embed(tokens, c.dtype, ex->fw[0].attn_norm, tp, dm, ex->ws, s));
  for (int l = 0; l < c.n_layers; ++l) {
    const FastWeights& w = ex->fw[l];
    cv.layer = l;
    HIP_TRY(launch_gemm_qkv(w, tp, dm, ex->ws, s, l > 0));
    HIP_TRY(launch_attention(cv, tp, dm, ex->ws, wpg, s, true));
    HIP_TRY(launch_combine(tp, dm, ex->ws, s, &cv));  // and the new rows, after the old ones were read
    HIP_TRY(launch_gemm_o(w, tp, dm, ex->ws, ks_o, s));
    HIP_TRY(launch_reduce_norm(tp, dm, ex->ws, ks_o, w.ffn_norm, nullptr, s));
    HIP_TRY(launch_gemm_gu(w, tp, dm, ex->ws, s));
    HIP_TRY(launch_gemm_down(w, tp, dm, ex->ws, ks_d, s));
    const float* gnext = l + 1 < c.n_layers ? ex->fw[l + 1].attn_norm : ex->final_norm;
    HIP_TRY(launch_reduce_norm(tp, dm, ex->ws, ks_d, gnext, hidden ? hidden + (int64_t)l * tp.M * dm.d : nullptr, s));
  }
  HIP_TRY(hipEventRecord(ex->done, s));
  for (int b = 0; b < batch; ++b) {  // the ring state after the append, as fsx_cache_append_rows
    const int64_t st = cache->len[b] > 0 ? cache->start[b] : first[b];
    const int64_t nl = cache->len[b] + n_rows;
    if (nl <= cache->capacity) {
      cache->start[b] = st;
      cache->len[b] = nl;
    } else {
      cache->start[b] = (st + (nl - cache->capacity)) % cache->capacity;
      cache->len[b] = cache->capacity;
    }
    cache->pos[b] += n_rows;
  }
  g_err.clear();
  return FSX_OK;
}

extern "C" int fsx_backbone_info(const fsx_backbone* bb, int64_t* weight_bytes, int64_t* workspace_bytes) {
  if (!bb || !bb->ex) return fail(FSX_E_INVALID, "backbone handle is NULL");
  if (weight_bytes) *weight_bytes = bb->ex->weight_bytes;
  if (workspace_bytes) *workspace_bytes = bb->ex->ws_bytes;
  return FSX_OK;
}

extern "C" void fsx_backbone_destroy(fsx_backbone* bb) {
  if (!bb) return;
  fsx_expert_destroy(bb->ex);
  delete bb;
}
