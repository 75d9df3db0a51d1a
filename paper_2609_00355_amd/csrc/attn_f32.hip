// Split-KV attention for the block draft and the ancestor-masked tree verify,
// fp32 in / fp32 out, on the vector ALUs.  Same work decomposition and
// partial-result format as the bf16 matrix-core kernel; meant for the small
// fp32 shapes in which exactness is decided (the paper audits losslessness in
// fp32, Sec. 3.3 and App. C).
//
// One workgroup owns (sequence b, KV head g, context split s, 32-row group).
// K/V tiles of 64 keys are staged in LDS.  A wave scores the 64 keys
// (lane = key) against its 8 rows' queries held in LDS, the 8 dot products
// side by side, updates each row's running max and sum (online softmax, exp2
// domain; the row maximum by a DPP reduction), writes the probabilities to
// LDS and accumulates P.V with lane = dim, again 8 rows side by side.  Each
// row's sums keep the order of a plain loop (dims, then keys, ascending).
// Global reads are 16-byte loads (the host requires 16-byte aligned tensors
// and rows of 64 or 128 floats), all of a tile's issued before any is used,
// and the next tile's are in flight while the current one is computed; the
// tree's parents are read once into LDS and walked there.
#include "glance_internal.h"

namespace glance {
namespace {

constexpr float kNegInf = -__builtin_inff();

// Maximum over the wave, returned uniform: butterflies within 16-lane rows,
// then row_bcast:15 / row_bcast:31 fold the rows into lane 63 (all lanes
// active; lanes a row mask leaves out keep their value, neutral for a max).
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, v),
                                                               __builtin_bit_cast(int, v), CTRL, ROWS, 0xf, false));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<0xb1, 0xf>(v));   // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_f<0x4e, 0xf>(v));   // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_f<0x141, 0xf>(v));  // row_half_mirror
  v = fmaxf(v, dpp_f<0x140, 0xf>(v));  // row_mirror
  v = fmaxf(v, dpp_f<0x142, 0xa>(v));  // row_bcast:15
  v = fmaxf(v, dpp_f<0x143, 0xc>(v));  // row_bcast:31
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
// Sum over the wave, the same way (lanes a row mask leaves out add 0).
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_z(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROWS, 0xf, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_z<0xb1, 0xf>(v);
  v += dpp_z<0x4e, 0xf>(v);
  v += dpp_z<0x141, 0xf>(v);
  v += dpp_z<0x140, 0xf>(v);
  v += dpp_z<0x142, 0xa>(v);
  v += dpp_z<0x143, 0xc>(v);
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

template <int D, bool TREE>
__global__ __launch_bounds__(kWaves * 64) void attn_f32_partial(AttnParams p) {
  constexpr int RPW = kF32RowsPerWave;
  constexpr int RB = kF32RowBlock;
  constexpr int DPL = D / 64;  // output dims per lane
  __shared__ float sK[kKeyTile * (D + 1)];  // +1: lanes read different keys at the same dim
  __shared__ __attribute__((aligned(16))) float sV[kKeyTile * D];
  __shared__ __attribute__((aligned(16))) float sQ[RB * D];
  __shared__ __attribute__((aligned(16))) float sP[kWaves][RPW][kKeyTile];
  __shared__ unsigned long long sAnc[64];
  __shared__ int sPar[64];

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

  // query rows of this row group (zeros for padding rows), 16 bytes a load
  constexpr int D4 = D / 4;
  constexpr int QPER = RB * D4 / (kWaves * 64);
  static_assert(RB * D4 % (kWaves * 64) == 0, "whole float4s per thread");
  float4 qv[QPER];
#pragma unroll
  for (int i = 0; i < QPER; ++i) {
    const int e = tid + i * kWaves * 64;
    const int lrow = e / D4;
    const int row = rg * RB + lrow;
    qv[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (row < p.rows) {
      const int node = row / p.group;
      const int hl = row - node * p.group;
      qv[i] = reinterpret_cast<const float4*>(q + (((size_t)b * p.n + node) * p.hq + (size_t)g * p.group + hl) * D)[e - lrow * D4];
    }
  }
  int par = -1;
  if (TREE && has_new && tid < p.n) par = p.parents[(size_t)b * p.n + tid];

  float o[RPW][DPL], m_run[RPW], l_run[RPW];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    m_run[r] = kNegInf;
    l_run[r] = 0.f;
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[r][i] = 0.f;
  }
  const float c = p.scale_log2;

  // tile t's K and V rows, 16 bytes a load, into registers (rows past the
  // tile's valid keys read as zeros)
  constexpr int TPER = kKeyTile * D4 / (kWaves * 64);
  static_assert(kKeyTile * D4 % (kWaves * 64) == 0, "whole float4s per thread");
  float4 kr[TPER], vr[TPER];
  auto load_tile = [&](int t, int& nvalid) {
    const bool is_new = (t == n_ctx_tiles);
    const float* kb;
    const float* vb;
    size_t stride;
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
#pragma unroll
    for (int i = 0; i < TPER; ++i) {
      const int e = tid + i * kWaves * 64;
      const int key = e / D4;
      const int d4 = e - key * D4;
      kr[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      vr[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (key < nvalid) {
        kr[i] = reinterpret_cast<const float4*>(kb + key * stride)[d4];
        vr[i] = reinterpret_cast<const float4*>(vb + key * stride)[d4];
      }
    }
  };
  // The first tile's loads go out with the query's and the parents', so that
  // one memory round trip brings all three.
  int nv_next = 0;
  if (n_tiles > 0) load_tile(0, nv_next);
  if (TREE && has_new && tid < p.n) sPar[tid] = par;
#pragma unroll
  for (int i = 0; i < QPER; ++i) reinterpret_cast<float4*>(sQ)[tid + i * kWaves * 64] = qv[i];
  __syncthreads();
  // ancestor-or-self word of each tree node, walked in LDS
  if (TREE && has_new && tid < p.n) {
    unsigned long long a = 1ull << tid;
    int cur = tid;
    int c = sPar[tid];
    for (int step = 0; step < 64 && c >= 0 && c < cur; ++step) {
      a |= 1ull << c;
      cur = c;
      c = sPar[c];
    }
    sAnc[tid] = a;
  }
  for (int t = 0; t < n_tiles; ++t) {
    const bool is_new = (t == n_ctx_tiles);
    const int nvalid = nv_next;
    __syncthreads();  // previous tile fully consumed
#pragma unroll
    for (int i = 0; i < TPER; ++i) {
      const int e = tid + i * kWaves * 64;
      const int key = e / D4;
      const int dd = 4 * (e - key * D4);
      float* kd = sK + key * (D + 1) + dd;
      kd[0] = kr[i].x;
      kd[1] = kr[i].y;
      kd[2] = kr[i].z;
      kd[3] = kr[i].w;
      *reinterpret_cast<float4*>(sV + key * D + dd) = vr[i];
    }
    __syncthreads();
    if (t + 1 < n_tiles) load_tile(t + 1, nv_next);  // in flight during this tile

    // scores of the wave's rows, lane = key: the rows' dot products run side
    // by side (each in its own order of dims), reading four query dims of a
    // row per 16-byte broadcast
    float sc[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) sc[r] = 0.f;
    const float4* q4 = reinterpret_cast<const float4*>(sQ) + wave * RPW * (D / 4);
#pragma unroll 2
    for (int d4 = 0; d4 < D / 4; ++d4) {
      const float* kp = sK + lane * (D + 1) + 4 * d4;
      const float k0 = kp[0], k1 = kp[1], k2 = kp[2], k3 = kp[3];
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        const float4 qv4 = q4[r * (D / 4) + d4];
        sc[r] = fmaf(qv4.x, k0, sc[r]);
        sc[r] = fmaf(qv4.y, k1, sc[r]);
        sc[r] = fmaf(qv4.z, k2, sc[r]);
        sc[r] = fmaf(qv4.w, k3, sc[r]);
      }
    }
    // softmax update of each row
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int row = rg * RB + wave * RPW + r;
      bool vis = lane < nvalid;
      if (TREE && is_new) {
        const int node = row < p.rows ? row / p.group : p.n;
        const unsigned long long anc = node < p.n ? sAnc[node] : ~0ull;
        vis = vis && ((anc >> lane) & 1ull);
      }
      const float sv = vis ? sc[r] : kNegInf;
      const float m_new = fmaxf(m_run[r], wave_max(sv));
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
    // P.V, lane = output dim: the rows side by side, four keys' probabilities
    // of a row per 16-byte broadcast
    float acc[RPW][DPL];
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
      for (int i = 0; i < DPL; ++i) acc[r][i] = 0.f;
#pragma unroll 2
    for (int k4 = 0; k4 < kKeyTile / 4; ++k4) {
      float v[4][DPL];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int i = 0; i < DPL; ++i) v[u][i] = sV[(4 * k4 + u) * D + lane + 64 * i];
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        const float4 p4 = reinterpret_cast<const float4*>(sP[wave][r])[k4];
#pragma unroll
        for (int i = 0; i < DPL; ++i) {
          acc[r][i] = fmaf(p4.x, v[0][i], acc[r][i]);
          acc[r][i] = fmaf(p4.y, v[1][i], acc[r][i]);
          acc[r][i] = fmaf(p4.z, v[2][i], acc[r][i]);
          acc[r][i] = fmaf(p4.w, v[3][i], acc[r][i]);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
      for (int i = 0; i < DPL; ++i) o[r][i] += acc[r][i];
  }

#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const float l = wave_sum(l_run[r]);
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
