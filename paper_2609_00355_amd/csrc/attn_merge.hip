// Second pass of split-KV attention: combine the per-split partial results.
//
// Each split s of a row left (m_s, l_s, O_s) with m_s the split's running
// maximum of the scaled scores in log2 units, l_s = sum exp2(score - m_s) and
// O_s = sum exp2(score - m_s) v (unnormalised).  With M = max_s m_s:
//   out = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s,   lse = (M + log2 L) ln 2
// One wave per output row; the row index is the output's own
// (b, new row, query head) index, so writes are contiguous.
#include "glance_internal.h"

namespace glance {
namespace {

constexpr float kLn2 = 0.6931471805599453f;

template <int D, bool BF16>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p) {
  constexpr int DPL = D / 64;
  const int lane = threadIdx.x & 63;
  const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const long total = (long)p.batch * p.n * p.hq;
  if (row >= total) return;
  const int h = (int)(row % p.hq);
  const long bi = row / p.hq;
  const int i = (int)(bi % p.n);
  const int b = (int)(bi / p.n);
  const int g = h / p.group;
  const int r = i * p.group + (h - g * p.group);

  int ctx = p.ctx_lens[b];
  ctx = ctx < 0 ? 0 : (ctx > p.cap ? p.cap : ctx);
  const int nsb = ctx > 0 ? (ctx + p.split_keys - 1) / p.split_keys : 1;

  const size_t base = ((size_t)b * p.hkv + g) * p.nsplit * p.rows_pad + r;
  // pass 1: the largest split maximum, lanes striding over the splits
  float M = -__builtin_inff();
  for (int s = lane; s < nsb; s += 64) M = fmaxf(M, p.part_ml[base + (size_t)s * p.rows_pad].x);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  // pass 2: lane s of each 64-split chunk computes the weight of split s; the
  // weights are broadcast while every lane accumulates its own output dims,
  // with the partial loads of several splits in flight at once.
  float lsum = 0.f;
  float acc[DPL];
#pragma unroll
  for (int k = 0; k < DPL; ++k) acc[k] = 0.f;
  for (int s0 = 0; s0 < nsb; s0 += 64) {
    float w = 0.f;
    if (s0 + lane < nsb) {
      const float2 ml = p.part_ml[base + (size_t)(s0 + lane) * p.rows_pad];
      w = exp2f(ml.x - M);
      lsum = fmaf(w, ml.y, lsum);
    }
    const int cnt = min(64, nsb - s0);
    for (int k0 = 0; k0 < cnt; k0 += 8) {
      float wk[8], v[8][DPL];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int k = k0 + u;
        wk[u] = __shfl(w, k & 63);  // 0 past the last split
        const float* po = p.part_o + (base + (size_t)(s0 + k) * p.rows_pad) * D + lane * DPL;
#pragma unroll
        for (int e = 0; e < DPL; ++e) v[u][e] = k < cnt ? po[e] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[e] = fmaf(wk[u], v[u][e], acc[e]);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) lsum += __shfl_xor(lsum, off);
  const float inv = 1.f / lsum;
  if (BF16) {
    __bf16* out = static_cast<__bf16*>(p.out) + row * D + lane * DPL;
#pragma unroll
    for (int k = 0; k < DPL; ++k) out[k] = (__bf16)(acc[k] * inv);
  } else {
    float* out = static_cast<float*>(p.out) + row * D + lane * DPL;
#pragma unroll
    for (int k = 0; k < DPL; ++k) out[k] = acc[k] * inv;
  }
  if (p.lse && lane == 0) p.lse[row] = (M + log2f(lsum)) * kLn2;
}

}  // namespace

hipError_t launch_attn_merge(const AttnParams& p, bool out_bf16, hipStream_t s) {
  const long total = (long)p.batch * p.n * p.hq;
  const dim3 grid((unsigned)((total + 3) / 4)), block(256);
  if (p.d == 128) {
    if (out_bf16) hipLaunchKernelGGL((attn_merge_kernel<128, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_merge_kernel<128, false>), grid, block, 0, s, p);
  } else {
    if (out_bf16) hipLaunchKernelGGL((attn_merge_kernel<64, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_merge_kernel<64, false>), grid, block, 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace glance
