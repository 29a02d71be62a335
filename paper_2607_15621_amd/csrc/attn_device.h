// Split-K joint attention of one work item (Eq. (1)), shared by the per-phase kernels and the tick kernel.
//
// A work item is (agent b, head h, a range of rows, a tile of 16 queries).  Per 32-row tile:
//   S^T = K Q^T on MFMA (A operand: 16 rows x 32 channels straight from memory in 16-byte loads; B operand:
//   the 16 queries, kept in registers); scores arrive in log2 units (q is pre-scaled by log2(e)/sqrt(Dh));
//   online softmax with the row max reduced over the 4 lanes sharing a query (xor 16, xor 32);
//   P (bf16/f16) is re-used in place as the A operand of O += P V: the lane's own 8 scores are rows
//   {4g..4g+3, 16+4g..16+4g+3}, and V is loaded as exactly those 8 rows x 8 channels per lane (each load
//   instruction reads 4 whole 256-byte rows) and transposed 8x8 in registers, so MFMA k (k = 0..7)
//   produces output channels 8c + k.
// The item writes its unnormalised output, running max (log2 units) and sum.  fp8 rows are decoded to
// fp16 in registers (exact) and use fp16 MFMA; the per-(agent, layer, head) scales multiply the scores
// (keys) and the partial output (values).
#pragma once

#include "common.h"

namespace fsx {

template <int KT, bool COH>  // KT 0: bf16 operands, 1: f16 operands
__device__ __forceinline__ void load_q_frag(const float* __restrict__ q, int64_t row, bool valid, int grp,
                                            uint4 qf[4]) {
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
    if (valid) {
      const float* p = q + row + 32 * kb + 8 * grp;
      lo = ldf4<COH>(p);
      hi = ldf4<COH>(p + 4);
    }
    if (KT == 0)
      qf[kb] = make_uint4(pack_bf16x2(lo.x, lo.y), pack_bf16x2(lo.z, lo.w), pack_bf16x2(hi.x, hi.y),
                          pack_bf16x2(hi.z, hi.w));
    else
      qf[kb] = make_uint4(pack_f16x2(lo.x, lo.y), pack_f16x2(lo.z, lo.w), pack_f16x2(hi.x, hi.y),
                          pack_f16x2(hi.z, hi.w));
  }
}

// 16-byte group of 8 consecutive channels of one row -> 8 x 16-bit MFMA operand values.
template <int KT, bool COH>
__device__ __forceinline__ uint4 load8(const char* p) {
  if constexpr (KT == 0) {
    return ld16<COH>(p);
  } else {
    const uint2 raw = *reinterpret_cast<const uint2*>(p);
    return make_uint4(e4m3x2_to_f16x2(raw.x, false), e4m3x2_to_f16x2(raw.x, true), e4m3x2_to_f16x2(raw.y, false),
                      e4m3x2_to_f16x2(raw.y, true));
  }
}

// rows i in [i0, i1) of one (agent, head): row i lives at base + slot(i) * row_bytes, where
// slot(i) = (start + i) mod cap for a ring and i for the expert's own rows.  The query of lane column c sees only
// rows i <= qmax0 + c (a causal mask among new rows; pass a large qmax0 for none).
// COH_ROWS: rows are read with device-coherent loads (rows produced inside the same launch);
// COH_OUT: the partial is written with device-coherent stores (consumed inside the same launch).
template <int KT, bool RING, bool COH_ROWS, bool COH_OUT>
__device__ void attn_rows(const char* __restrict__ kbase, const char* __restrict__ vbase, int64_t row_bytes,
                          int64_t start, int64_t cap, int i0, int i1, const uint4 qf[4], float kscale, float vscale,
                          int lane, float* __restrict__ out_o, float* __restrict__ out_ml, int Dh,
                          int qmax0 = 1 << 30) {
  constexpr int ES = KT == 0 ? 2 : 1;
  const int c = lane & 15, grp = lane >> 4;
  const int qmax = qmax0 + c;
  auto roff = [&](int i) -> int64_t {
    int64_t slot = i;
    if (RING) {
      slot = start + i;
      if (slot >= cap) slot -= cap;
    }
    return slot * row_bytes;
  };
  f32x4 o[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) o[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  for (int r0 = i0; r0 < i1; r0 += 32) {
    uint4 kf[2][4];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int i = r0 + 16 * rt + c;
      const char* p = kbase + roff(i < i1 ? i : i0);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) kf[rt][kb] = load8<KT, COH_ROWS>(p + (32 * kb + 8 * grp) * ES);
    }
    uint4 vr[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int rr = r0 + (j < 4 ? 4 * grp + j : 16 + 4 * grp + (j - 4));
      vr[j] = load8<KT, COH_ROWS>(vbase + roff(rr < i1 ? rr : i0) + 8 * c * ES);
    }
    f32x4 s[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      s[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        s[rt] = KT == 0 ? mfma_bf16(kf[rt][kb], qf[kb], s[rt]) : mfma_f16(kf[rt][kb], qf[kb], s[rt]);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rr = r0 + 16 * rt + 4 * grp + i;
        const float v = rr < i1 && rr <= qmax ? s[rt][i] * kscale : -INFINITY;
        s[rt][i] = v;
        mx = fmaxf(mx, v);
      }
    mx = rows_max(mx);
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
    if (KT == 0)
      pf = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                      pack_bf16x2(p[6], p[7]));
    else
      pf = make_uint4(pack_f16x2(p[0], p[1]), pack_f16x2(p[2], p[3]), pack_f16x2(p[4], p[5]), pack_f16x2(p[6], p[7]));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a_i = col_pick(alpha, grp, i);
#pragma unroll
      for (int k = 0; k < 8; ++k) o[k][i] *= a_i;
    }
    uint4 vt[8];
    transpose8x8_b16(vr, vt);
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = KT == 0 ? mfma_bf16(pf, vt[k], o[k]) : mfma_f16(pf, vt[k], o[k]);
  }
  const float lt = rows_sum(l_run);
  if (grp == 0) {
    stf<COH_OUT>(out_ml + c * 2 + 0, m_run);
    stf<COH_OUT>(out_ml + c * 2 + 1, lt);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float* dst = out_o + (4 * grp + i) * Dh + 8 * c;
    stf4<COH_OUT>(dst, make_float4(o[0][i] * vscale, o[1][i] * vscale, o[2][i] * vscale, o[3][i] * vscale));
    stf4<COH_OUT>(dst + 4, make_float4(o[4][i] * vscale, o[5][i] * vscale, o[6][i] * vscale, o[7][i] * vscale));
  }
}

}  // namespace fsx
