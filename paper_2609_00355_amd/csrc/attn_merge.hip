// Second pass of split-KV attention: combine the per-split partial results.
//
// Each split s of a row left (m_s, l_s, O_s) with m_s the split's running
// maximum of the scaled scores in log2 units, l_s = sum exp2(score - m_s) and
// O_s = sum exp2(score - m_s) v (unnormalised).  With M = max_s m_s:
//   out = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s,   lse = (M + log2 L) ln 2
//
// attn_merge_kernel (fp32 attention): D/4 lanes serve one output row, four
// dims (16 bytes) each, so a wave merges 64/(D/4) rows.  The row index is the
// output's own (b, new row, query head) index, so writes are contiguous.  The
// (m, l) pairs and the O partials of up to kChunk splits are loaded together,
// before any of them is needed, so a row with at most kChunk splits costs one
// memory round trip; longer rows take further chunks, rescaled online like
// the attention itself.
//
// attn_merge_pieces (bf16 attention): the partials are the pieces' MFMA
// register tiles in fp16, each row scaled by a power of two that the row's
// (max, sum) pair carries (lane l of a 32-row tile holds row l % 32 and, in
// quad k, dims 32 (k / 4) + 8 (k % 4) + 4 (l / 32) .. +3).  A thread owns one
// (row, four dims) and reads that quad of every piece of its sequence, in
// piece order, all loads of a chunk of 16 pieces issued before any is used;
// consecutive threads read consecutive lanes, 512 bytes per wave-wide load.
// Sequences with one piece were written by the attention kernel and are
// skipped.
#include "glance_internal.h"

namespace glance {
namespace {

constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMergeWaves = 2;
typedef __attribute__((ext_vector_type(4))) _Float16 f16x4;

template <int D, bool BF16>
__global__ __launch_bounds__(64 * kMergeWaves) void attn_merge_kernel(AttnParams p) {
  constexpr int LPR = D / 4;     // lanes per row
  constexpr int RPW = 64 / LPR;  // rows per wave
  constexpr int kChunk = 16;     // splits in flight per lane
  static_assert(kChunk <= LPR, "one (m, l) pair per lane and chunk");
  const int lane = threadIdx.x & 63;
  const int q = lane % LPR;
  const int lead = lane - q;  // first lane of this row
  // row counts are far below 2^31 (batch * new rows * query heads), so 32-bit index math
  const int total = p.batch * p.n * p.hq;
  const int row_raw = ((int)blockIdx.x * kMergeWaves + (int)(threadIdx.x >> 6)) * RPW + lane / LPR;
  const bool live = row_raw < total;
  const int row = live ? row_raw : total - 1;  // dead lanes shadow the last row, store nothing
  const int h = (unsigned)row % (unsigned)p.hq;
  const int bi = (unsigned)row / (unsigned)p.hq;
  const int i = (unsigned)bi % (unsigned)p.n;
  const int b = (unsigned)bi / (unsigned)p.n;
  const int g = h / p.group;
  const int r = i * p.group + (h - g * p.group);

  int ctx = p.ctx_lens[b];
  ctx = ctx < 0 ? 0 : (ctx > p.cap ? p.cap : ctx);
  const int nsb = ctx > 0 ? (ctx + p.split_keys - 1) / p.split_keys : 1;

  const size_t base = ((size_t)b * p.hkv + g) * p.nsplit * p.rows_pad + r;
  const float4* po = reinterpret_cast<const float4*>(p.part_o) + base * (D / 4) + q;
  const size_t sstride = (size_t)p.rows_pad * (D / 4);  // float4s from one split to the next

  float M = -__builtin_inff();
  float lsum = 0.f;  // this lane's share of the denominator
  float4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < nsb; s0 += kChunk) {
    const int cnt = min(kChunk, nsb - s0);
    float2 ml = {-__builtin_inff(), 0.f};
    if (q < cnt) ml = p.part_ml[base + (size_t)(s0 + q) * p.rows_pad];
    float4 v[kChunk];
#pragma unroll
    for (int u = 0; u < kChunk; ++u)
      v[u] = u < cnt ? po[(size_t)(s0 + u) * sstride] : float4{0.f, 0.f, 0.f, 0.f};
    float mc = ml.x;
#pragma unroll
    for (int off = LPR / 2; off >= 1; off >>= 1) mc = fmaxf(mc, __shfl_xor(mc, off));
    const float Mn = fmaxf(M, mc);
    const float sc = M == -__builtin_inff() ? 0.f : exp2f(M - Mn);
    const float w = q < cnt ? exp2f(ml.x - Mn) : 0.f;
    lsum = fmaf(w, ml.y, lsum * sc);
    acc.x *= sc; acc.y *= sc; acc.z *= sc; acc.w *= sc;
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const float wu = __shfl(w, lead + u);  // 0 past the last split
      acc.x = fmaf(wu, v[u].x, acc.x);
      acc.y = fmaf(wu, v[u].y, acc.y);
      acc.z = fmaf(wu, v[u].z, acc.z);
      acc.w = fmaf(wu, v[u].w, acc.w);
    }
    M = Mn;
  }
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1) lsum += __shfl_xor(lsum, off);
  if (!live) return;
  const float inv = 1.f / lsum;
  if (BF16) {
    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
    const bf16x4 o = {(__bf16)(acc.x * inv), (__bf16)(acc.y * inv), (__bf16)(acc.z * inv),
                      (__bf16)(acc.w * inv)};
    *reinterpret_cast<bf16x4*>(static_cast<__bf16*>(p.out) + (size_t)row * D + 4 * q) = o;
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(p.out) + (size_t)row * D + 4 * q) =
        float4{acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv};
  }
  if (p.lse && q == 0) p.lse[row] = (M + log2f(lsum)) * kLn2;
}


template <int D>
__global__ __launch_bounds__(256) void attn_merge_pieces(AttnParams p) {
  constexpr int KQ = D / 8;    // quads of values per lane of a tile (OV / 4)
  constexpr int WG_K = 4;      // quad slots per workgroup (one per wave)
  constexpr int kChunk = 16;
  const int lane = threadIdx.x & 63;
  const int k = (blockIdx.x % (KQ / WG_K)) * WG_K + (threadIdx.x >> 6);
  int unit = blockIdx.x / (KQ / WG_K);  // ((b * hkv + g) * row_groups + rgi) * tiles_rg + w
  const int w = unit % p.tiles_rg;
  unit /= p.tiles_rg;
  const int rgi = unit % p.row_groups;
  unit /= p.row_groups;
  const int g = unit % p.hkv;
  const int b = unit / p.hkv;
  const int2 pl = p.plan[b];  // (pieces, first slot)
  if (pl.x <= 1) return;
  const int r32 = lane & 31, h = lane >> 5;
  const int row = 32 * (rgi * p.tiles_rg + w) + r32;
  if (row >= p.rows) return;
  const int node = row / p.group;
  const size_t out_row = ((size_t)b * p.n + node) * p.hq + (size_t)g * p.group + (row - node * p.group);
  const int d0 = 32 * (k >> 2) + 8 * (k & 3) + 4 * h;

  const size_t ws0 = ((size_t)g * p.slots_per_g + pl.y) * p.row_groups + rgi;  // piece q: ws0 + q * row_groups
  const size_t o_stride = (size_t)p.row_groups * p.tiles_rg * KQ * 64;          // fp16 quads between pieces
  const size_t ml_stride = (size_t)p.row_groups * p.rows_rg;
  const f16x4* po = reinterpret_cast<const f16x4*>(p.part_o) + (ws0 * p.tiles_rg + w) * KQ * 64 + k * 64 + lane;
  const float2* pm = p.part_ml + ws0 * p.rows_rg + 32 * w + r32;

  float M = -__builtin_inff(), lsum = 0.f;
  float4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int q0 = 0; q0 < pl.x; q0 += kChunk) {
    const int cnt = min(kChunk, pl.x - q0);
    float2 ml[kChunk];
    f16x4 v[kChunk];
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      ml[u] = u < cnt ? pm[(size_t)(q0 + u) * ml_stride] : make_float2(-__builtin_inff(), 0.f);
      v[u] = u < cnt ? po[(size_t)(q0 + u) * o_stride] : f16x4{};
    }
    float mc = M;
#pragma unroll
    for (int u = 0; u < kChunk; ++u) mc = fmaxf(mc, ml[u].x);
    const float sc = M == -__builtin_inff() ? 0.f : exp2f(M - mc);
    lsum *= sc;
    acc.x *= sc; acc.y *= sc; acc.z *= sc; acc.w *= sc;
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const float wu = u < cnt ? exp2f(ml[u].x - mc) : 0.f;
      lsum = fmaf(wu, ml[u].y, lsum);
      acc.x = fmaf(wu, (float)v[u][0], acc.x);
      acc.y = fmaf(wu, (float)v[u][1], acc.y);
      acc.z = fmaf(wu, (float)v[u][2], acc.z);
      acc.w = fmaf(wu, (float)v[u][3], acc.w);
    }
    M = mc;
  }
  const float inv = 1.f / lsum;
  typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
  const bf16x4 o = {(__bf16)(acc.x * inv), (__bf16)(acc.y * inv), (__bf16)(acc.z * inv), (__bf16)(acc.w * inv)};
  *reinterpret_cast<bf16x4*>(static_cast<__bf16*>(p.out) + out_row * D + d0) = o;
  if (p.lse && k == 0 && h == 0) p.lse[out_row] = (M + log2f(lsum)) * kLn2;
}

}  // namespace

hipError_t launch_attn_merge_pieces(const AttnParams& p, hipStream_t s) {
  const long units = (long)p.batch * p.hkv * p.row_groups * p.tiles_rg;
  const dim3 grid((unsigned)(units * (p.d / 8) / 4)), block(256);
  if (p.d == 128) hipLaunchKernelGGL((attn_merge_pieces<128>), grid, block, 0, s, p);
  else hipLaunchKernelGGL((attn_merge_pieces<64>), grid, block, 0, s, p);
  return hipGetLastError();
}

hipError_t launch_attn_merge(const AttnParams& p, bool out_bf16, hipStream_t s) {
  const long total = (long)p.batch * p.n * p.hq;
  const long rows_per_wg = (long)kMergeWaves * 64 / (p.d / 4);
  const dim3 grid((unsigned)((total + rows_per_wg - 1) / rows_per_wg)), block(64 * kMergeWaves);
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
