// Split-KV attention for the block draft and the ancestor-masked tree verify,
// fp32 in / fp32 out, on the vector ALUs.  Same work decomposition and
// partial-result format as the bf16 matrix-core kernel; meant for the small
// fp32 shapes in which exactness is decided (the paper audits losslessness in
// fp32, Sec. 3.3 and App. C).
//
// One workgroup owns (sequence b, KV head g, context split s, 32-row group).
// K/V tiles of 64 keys are staged in LDS.  For each of its 8 rows a wave
//   scores the 64 keys (lane = key) against the row's query held in LDS,
//   updates the row's running max and sum (online softmax, exp2 domain),
//   writes the 64 probabilities to LDS and accumulates P.V with lane = dim.
#include "glance_internal.h"

namespace glance {
namespace {

constexpr float kNegInf = -__builtin_inff();

template <int D, bool TREE>
__global__ __launch_bounds__(kWaves * 64) void attn_f32_partial(AttnParams p) {
  constexpr int RPW = kF32RowsPerWave;
  constexpr int RB = kF32RowBlock;
  constexpr int DPL = D / 64;  // output dims per lane
  __shared__ float sK[kKeyTile * (D + 1)];  // +1: lanes read different keys at the same dim
  __shared__ float sV[kKeyTile * D];
  __shared__ float sQ[RB * D];
  __shared__ float sP[kWaves][RPW][kKeyTile];
  __shared__ unsigned long long sAnc[64];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar branches

  const int L = blockIdx.x;
  const int xcd = L & 7;
  const int q8 = L >> 3;
  const int rg = q8 % p.row_groups;
  const int grp = (q8 / p.row_groups) * 8 + xcd;
  if (grp >= p.nsplit * p.batch * p.hkv) return;
  const int g = grp % p.hkv;
  const int bs = grp / p.hkv;
  const int b = bs % p.batch;
  const int s = bs / p.batch;

  int ctx = p.ctx_lens[b];
  ctx = ctx < 0 ? 0 : (ctx > p.cap ? p.cap : ctx);
  const int nsb = ctx > 0 ? (ctx + p.split_keys - 1) / p.split_keys : 1;
  if (s >= nsb) return;
  const int k_begin = s * p.split_keys;
  const int k_end = min(ctx, k_begin + p.split_keys);
  const bool has_new = (s == nsb - 1);
  const int n_ctx_tiles = k_end > k_begin ? (k_end - k_begin + kKeyTile - 1) / kKeyTile : 0;
  const int n_tiles = n_ctx_tiles + (has_new ? 1 : 0);

  const float* q = static_cast<const float*>(p.q);
  const float* kc = static_cast<const float*>(p.k_ctx);
  const float* vc = static_cast<const float*>(p.v_ctx);
  const float* kn = static_cast<const float*>(p.k_new);
  const float* vn = static_cast<const float*>(p.v_new);

  if (TREE && has_new && tid < p.n) {
    const int32_t* par = p.parents + (size_t)b * p.n;
    unsigned long long a = 1ull << tid;
    int cur = tid;
    int c = par[tid];
    for (int step = 0; step < 64 && c >= 0 && c < cur; ++step) {
      a |= 1ull << c;
      cur = c;
      c = par[c];
    }
    sAnc[tid] = a;
  }
  // Query rows of this row group (zeros for padding rows).
  for (int e = tid; e < RB * D; e += kWaves * 64) {
    const int lrow = e / D;
    const int dd = e - lrow * D;
    const int row = rg * RB + lrow;
    float v = 0.f;
    if (row < p.rows) {
      const int node = row / p.group;
      const int hl = row - node * p.group;
      v = q[(((size_t)b * p.n + node) * p.hq + (size_t)g * p.group + hl) * D + dd];
    }
    sQ[e] = v;
  }

  float o[RPW][DPL], m_run[RPW], l_run[RPW];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    m_run[r] = kNegInf;
    l_run[r] = 0.f;
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[r][i] = 0.f;
  }
  const float c = p.scale_log2;

  for (int t = 0; t < n_tiles; ++t) {
    const bool is_new = (t == n_ctx_tiles);
    const float* kb;
    const float* vb;
    size_t stride;
    int nvalid;
    if (!is_new) {
      const int key0 = k_begin + t * kKeyTile;
      nvalid = min(kKeyTile, k_end - key0);
      const size_t off = (((size_t)b * p.hkv + g) * p.cap + key0) * D;
      kb = kc + off;
      vb = vc + off;
      stride = D;
    } else {
      nvalid = p.n;
      const size_t off = ((size_t)b * p.n * p.hkv + g) * D;
      kb = kn + off;
      vb = vn + off;
      stride = (size_t)p.hkv * D;
    }
    __syncthreads();  // previous tile fully consumed
    for (int e = tid; e < kKeyTile * D; e += kWaves * 64) {
      const int key = e / D;
      const int dd = e - key * D;
      float kv = 0.f, vv = 0.f;
      if (key < nvalid) {
        kv = kb[key * stride + dd];
        vv = vb[key * stride + dd];
      }
      sK[key * (D + 1) + dd] = kv;
      sV[key * D + dd] = vv;
    }
    __syncthreads();

    // scores and softmax update, lane = key
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int lrow = wave * RPW + r;
      const int row = rg * RB + lrow;
      const float* qr = sQ + lrow * D;
      float sacc = 0.f;
#pragma unroll 8
      for (int dd = 0; dd < D; ++dd) sacc = fmaf(qr[dd], sK[lane * (D + 1) + dd], sacc);
      bool vis = lane < nvalid;
      if (TREE && is_new) {
        const int node = row < p.rows ? row / p.group : p.n;
        const unsigned long long anc = node < p.n ? sAnc[node] : ~0ull;
        vis = vis && ((anc >> lane) & 1ull);
      }
      const float sv = vis ? sacc : kNegInf;
      float mx = sv;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
      const float m_new = fmaxf(m_run[r], mx);
      const float m_use = (m_new == kNegInf) ? 0.f : m_new;
      const float alpha = exp2f((m_run[r] - m_use) * c);
      m_run[r] = m_new;
      const float e = exp2f(fmaf(sv, c, -m_use * c));
      l_run[r] = l_run[r] * alpha + e;  // per-lane partial sum; alpha is uniform over the row
      sP[wave][r][lane] = e;
#pragma unroll
      for (int i = 0; i < DPL; ++i) o[r][i] *= alpha;
    }
    __syncthreads();
    // P.V, lane = output dim
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      float acc[DPL];
#pragma unroll
      for (int i = 0; i < DPL; ++i) acc[i] = 0.f;
      for (int k = 0; k < kKeyTile; ++k) {
        const float pk = sP[wave][r][k];
#pragma unroll
        for (int i = 0; i < DPL; ++i) acc[i] = fmaf(pk, sV[k * D + lane + 64 * i], acc[i]);
      }
#pragma unroll
      for (int i = 0; i < DPL; ++i) o[r][i] += acc[i];
    }
  }

#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    float l = l_run[r];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) l += __shfl_xor(l, off);
    const int row = rg * RB + wave * RPW + r;
    const size_t pr = (((size_t)b * p.hkv + g) * p.nsplit + s) * p.rows_pad + row;
    if (lane == 0) p.part_ml[pr] = make_float2(m_run[r] * c, l);
#pragma unroll
    for (int i = 0; i < DPL; ++i) p.part_o[pr * D + lane + 64 * i] = o[r][i];
  }
}

}  // namespace

hipError_t launch_attn_f32(const AttnParams& p, bool tree, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const int groups = p.nsplit * p.batch * p.hkv;
  const dim3 grid(((groups + 7) / 8) * 8 * p.row_groups), block(kWaves * 64);
  if (ev0) (void)hipEventRecord(ev0, s);
  if (p.d == 128) {
    if (tree) hipLaunchKernelGGL((attn_f32_partial<128, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_f32_partial<128, false>), grid, block, 0, s, p);
  } else {
    if (tree) hipLaunchKernelGGL((attn_f32_partial<64, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_f32_partial<64, false>), grid, block, 0, s, p);
  }
  hipError_t e = hipGetLastError();
  if (ev1) (void)hipEventRecord(ev1, s);
  return e;
}

}  // namespace glance
