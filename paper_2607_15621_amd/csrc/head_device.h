// The paper's waypoint head (Sec. 3.1): the last n_queries expert tokens are learnable waypoint queries, each
// decoded to one (x, y) waypoint by a two-layer head -- final RMSNorm, Linear(d -> hidden) + bias, GELU (exact erf
// form), Linear(hidden -> 2) + bias.  One workgroup of 256 threads computes one agent; shared by the persistent tick
// kernel (which reads its tile-major residual) and the per-op paths (row-major residual).
#pragma once

#include "common.h"

namespace fsx {

constexpr int QH_MAX_QUERIES = 8;

struct QueryHead {
  const void* w1;   // [hidden][d] (wdtype)
  const float* b1;  // [hidden]
  const void* w2;   // [2][hidden] (wdtype)
  const float* b2;  // [2]
  int hidden;
  int wdtype;       // FSX_F32 or FSX_BF16
};

__device__ __forceinline__ float qh_weight(const void* w, int wdtype, int64_t i) {
  return wdtype == FSX_BF16 ? bf16_to_f32(reinterpret_cast<const uint16_t*>(w)[i]) : reinterpret_cast<const float*>(w)[i];
}

// row(t, col): residual of expert token t (0 <= t < T), column col.  out(o, v) stores output o (2q + {0: x, 1: y}).
// lds: nq * (d + hidden) floats.  Ends with a barrier; every thread of the workgroup must call it.
template <typename Row, typename Out>
__device__ void query_head_wg(Row row, int T, int nq, int d, float eps, const float* __restrict__ gfin,
                              const QueryHead& qh, Out out, float* lds) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, nw = blockDim.x >> 6;
  const int hid = qh.hidden;
  float* x = lds;           // [nq][d] normalised query rows
  float* hv = lds + nq * d; // [nq][hidden] hidden activations
  for (int i = tid; i < nq * d; i += blockDim.x) x[i] = row(T - nq + i / d, i % d);
  __syncthreads();
  for (int q = wave; q < nq; q += nw) {
    float ss = 0.f;
    for (int c = lane; c < d; c += WAVE) ss += x[q * d + c] * x[q * d + c];
    const float r = 1.0f / sqrtf(wave_sum(ss) / (float)d + eps);
    for (int c = lane; c < d; c += WAVE) x[q * d + c] *= r * gfin[c];
  }
  __syncthreads();
  // hidden unit j by one wave: lanes split the row of W1 (coalesced), one partial dot per query, summed across lanes
  for (int j = wave; j < hid; j += nw) {
    float acc[QH_MAX_QUERIES];
#pragma unroll
    for (int q = 0; q < QH_MAX_QUERIES; ++q) acc[q] = 0.f;
    for (int c = lane; c < d; c += WAVE) {
      const float w = qh_weight(qh.w1, qh.wdtype, (int64_t)j * d + c);
#pragma unroll
      for (int q = 0; q < QH_MAX_QUERIES; ++q)
        if (q < nq) acc[q] += w * x[q * d + c];
    }
#pragma unroll
    for (int q = 0; q < QH_MAX_QUERIES; ++q) {
      if (q < nq) {
        const float u = wave_sum(acc[q]) + qh.b1[j];
        if (lane == 0) hv[q * hid + j] = 0.5f * u * (1.0f + erff(u * 0.70710678118654752f));
      }
    }
  }
  __syncthreads();
  for (int o = wave; o < 2 * nq; o += nw) {
    const int q = o >> 1, cc = o & 1;
    float acc = 0.f;
    for (int j = lane; j < hid; j += WAVE) acc += qh_weight(qh.w2, qh.wdtype, (int64_t)cc * hid + j) * hv[q * hid + j];
    acc = wave_sum(acc) + qh.b2[cc];
    if (lane == 0) out(o, acc);
  }
  __syncthreads();
}

}  // namespace fsx
