// Split-KV attention for the block draft and the ancestor-masked tree verify,
// bf16 in / fp32 accumulate, on gfx950 matrix cores.
//
// One workgroup owns one (sequence b, KV head g, context split s, row group).
// Its rows are the flattened (new row, query head of the group) pairs, so the
// K/V tile staged in LDS is shared by every query head of the GQA group and
// by every block/tree row: the context is read from HBM once per split.
//
// Per 64-key LDS tile each wave computes, for each of its 16-row tiles,
//   S^T[key][row] = K[key][:] . Q[row][:]      (v_mfma_f32_16x16x32_bf16, A = K, B = Q^T)
//   online softmax over the keys of each row  (exp2 with the scale folded in)
//   O^T[d][row]  += V^T[d][key] . P^T[key][row] (A = V^T via ds_read_b64_tr_b16, B = P^T)
// S^T is computed with the key order permuted inside each 32-key group so
// that the MFMA result layout (lane l holds rows l%16, key slots 4*(l/16)+i)
// is directly the B operand of the P.V product (lane l needs 8 consecutive
// key slots 8*(l/16)..+7): no shuffle between the two contractions.
//
// The new keys (block or tree rows) are one extra tile processed by the last
// split of each sequence; for the tree, node i sees key j iff bit j of its
// ancestor word is set (Def. 1's packed verification).  Each split writes its
// unnormalised output and (max, sum) to the workspace; attn_merge.hip
// combines the splits.
#include "glance_internal.h"

namespace glance {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr float kNegInf = -__builtin_inff();

template <int D>
struct TileGeom {
  static constexpr int kStride = D + 8;  // bf16 per LDS key row: 16-byte pad against bank conflicts
  static constexpr int kChunks = D / 8;  // 16-byte chunks per key row
  static constexpr int kLoads = kKeyTile * kChunks / (kWaves * 64);  // chunks per thread per tensor
};

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int D, bool TREE>
__global__ __launch_bounds__(kWaves * 64) void attn_bf16_partial(AttnParams p) {
  constexpr int TPW = kBf16TilesPerWave;
  constexpr int KS = D / 32;  // k-steps of Q.K^T
  constexpr int DT = D / 16;  // d-tiles of P.V
  constexpr int ST = TileGeom<D>::kStride;
  constexpr int CH = TileGeom<D>::kChunks;
  constexpr int NL = TileGeom<D>::kLoads;
  static_assert(NL * kWaves * 64 == kKeyTile * CH, "tile load must divide evenly");

  __shared__ __attribute__((aligned(16))) __bf16 sK[2][kKeyTile * ST];
  __shared__ __attribute__((aligned(16))) __bf16 sV[2][kKeyTile * ST];
  __shared__ unsigned long long sAnc[64];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar branches
  const int lg = lane >> 4;   // lane group 0..3
  const int lr = lane & 15;   // row within a 16-row tile

  // ---- work item.  Blocks 8*(row_groups*j + r) + x form group 8*j + x, row
  // group r: the row groups sharing one KV split sit on the same XCD (block
  // index mod 8), so their repeated K/V reads hit that XCD's L2.
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
  if (s >= nsb) return;  // empty split of a shorter sequence
  const int k_begin = s * p.split_keys;
  const int k_end = min(ctx, k_begin + p.split_keys);
  const bool has_new = (s == nsb - 1);
  const int n_ctx_tiles = k_end > k_begin ? (k_end - k_begin + kKeyTile - 1) / kKeyTile : 0;
  const int n_tiles = n_ctx_tiles + (has_new ? 1 : 0);

  const __bf16* q = static_cast<const __bf16*>(p.q);
  const __bf16* kc = static_cast<const __bf16*>(p.k_ctx);
  const __bf16* vc = static_cast<const __bf16*>(p.v_ctx);
  const __bf16* kn = static_cast<const __bf16*>(p.k_new);
  const __bf16* vn = static_cast<const __bf16*>(p.v_new);

  // ---- ancestor words of the packed tree: anc[i] = {i} u anc[parent(i)].
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

  // ---- this wave's query rows, held as MFMA B operands for the whole split.
  const int tile0 = rg * (kWaves * TPW) + wave * TPW;
  const int n_row_tiles = (p.rows + 15) >> 4;
  bf16x8 qf[TPW][KS];
  int node_of[TPW];
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    const int row = (tile0 + j) * 16 + lr;
    node_of[j] = p.n;  // padding rows: treated as seeing every key
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[j][ks] = bf16x8{};
    if (row < p.rows) {
      const int node = row / p.group;
      const int hl = row - node * p.group;
      node_of[j] = node;
      const __bf16* qp = q + (((size_t)b * p.n + node) * p.hq + (size_t)g * p.group + hl) * D + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf[j][ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(qp + 32 * ks));
    }
  }

  f32x4 o[TPW][DT];
  float m_run[TPW], l_run[TPW];
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    m_run[j] = kNegInf;
    l_run[j] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[j][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float c = p.scale_log2;

  // ---- global -> register -> LDS staging, double buffered.
  u32x4 rk[NL], rv[NL];
  auto fetch = [&](int t) {
    const __bf16* kb;
    const __bf16* vb;
    size_t stride;
    int nvalid;
    if (t < n_ctx_tiles) {
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
    for (int i = 0; i < NL; ++i) {
      const int cidx = tid + i * kWaves * 64;
      const int key = cidx / CH;
      const int col = cidx % CH;
      if (key < nvalid) {
        rk[i] = *reinterpret_cast<const u32x4*>(kb + key * stride + col * 8);
        rv[i] = *reinterpret_cast<const u32x4*>(vb + key * stride + col * 8);
      } else {  // zero K and V outside the valid keys: P is 0 there and 0 * 0 stays 0
        rk[i] = u32x4{0u, 0u, 0u, 0u};
        rv[i] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int cidx = tid + i * kWaves * 64;
      const int key = cidx / CH;
      const int col = cidx % CH;
      *reinterpret_cast<u32x4*>(&sK[buf][key * ST + col * 8]) = rk[i];
      *reinterpret_cast<u32x4*>(&sV[buf][key * ST + col * 8]) = rv[i];
    }
  };

  auto compute = [&](int buf, int t) {
    const bool is_new = (t == n_ctx_tiles);
    const int nvalid = is_new ? p.n : min(kKeyTile, k_end - (k_begin + t * kKeyTile));
    const __bf16* Kt = sK[buf];
    const __bf16* Vt = sV[buf];

    // S^T = K Q^T for keys 32*kk + 8*lg' + 4*sub + (lane&3), lg' = (lane&15)>>2 on the A side.
    f32x4 sc[TPW][2][2];
#pragma unroll
    for (int j = 0; j < TPW; ++j)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) sc[j][kk][sub] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        const int krow = 32 * kk + 8 * (lr >> 2) + 4 * sub + (lane & 3);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 kop = as_bf16x8(*reinterpret_cast<const u32x4*>(Kt + krow * ST + 32 * ks + 8 * lg));
#pragma unroll
          for (int j = 0; j < TPW; ++j)
            if (tile0 + j < n_row_tiles)
              sc[j][kk][sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qf[j][ks], sc[j][kk][sub], 0, 0, 0);
        }
      }
    }

    // Mask, online softmax.  Result lane l holds row lr and keys 32*kk + 8*lg + 4*sub + i.
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      unsigned long long anc = ~0ull;
      if (TREE && is_new && node_of[j] < p.n) anc = sAnc[node_of[j]];
      float mx = kNegInf;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = 32 * kk + 8 * lg + 4 * sub + i;
            bool vis = key < nvalid;
            if (TREE && is_new) vis = vis && ((anc >> key) & 1ull);
            const float v = vis ? sc[j][kk][sub][i] : kNegInf;
            sc[j][kk][sub][i] = v;
            mx = fmaxf(mx, v);
          }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[j], mx);
      const float m_use = (m_new == kNegInf) ? 0.f : m_new;
      const float alpha = exp2f((m_run[j] - m_use) * c);
      m_run[j] = m_new;
      const float neg = -m_use * c;
      float lsum = 0.f;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float e = exp2f(fmaf(sc[j][kk][sub][i], c, neg));
            sc[j][kk][sub][i] = e;
            lsum += e;
          }
      l_run[j] = l_run[j] * alpha + lsum;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[j][dt] *= alpha;
    }

    // O^T += V^T P^T.  ds_read_b64_tr_b16: in each 16-lane group, lane jl reads
    // row key0 + (jl>>2), columns d0 + 4*(jl&3) .. +3, and receives
    // V[key0 + i][d0 + jl] for i = 0..3.
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8 pb[TPW];
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pb[j][i] = (__bf16)sc[j][kk][0][i];
          pb[j][4 + i] = (__bf16)sc[j][kk][1][i];
        }
      }
      const int vrow = 32 * kk + 8 * lg + (lr >> 2);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const __bf16* va = Vt + vrow * ST + 16 * dt + 4 * (lane & 3);
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(va));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(va + 4 * ST));
        // whole-vector reinterpretation: element-wise bf16 inserts of the 16-bit
        // lanes were miscompiled (every element became lo[0])
        const bf16x8 vop = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
        for (int j = 0; j < TPW; ++j)
          if (tile0 + j < n_row_tiles)
            o[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pb[j], o[j][dt], 0, 0, 0);
      }
    }
  };

  fetch(0);
  stash(0);
  __syncthreads();
  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < n_tiles) fetch(t + 1);
    compute(buf, t);
    if (t + 1 < n_tiles) stash(buf ^ 1);
    __syncthreads();
  }

  // ---- partial results of this split: O unnormalised, (max * c, sum).
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    if (tile0 + j >= n_row_tiles) continue;
    float l = l_run[j];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int row = (tile0 + j) * 16 + lr;
    const size_t pr = (((size_t)b * p.hkv + g) * p.nsplit + s) * p.rows_pad + row;
    if (lg == 0) p.part_ml[pr] = make_float2(m_run[j] * c, l);
    float* po = p.part_o + pr * D + 4 * lg;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) *reinterpret_cast<f32x4*>(po + 16 * dt) = o[j][dt];
  }
}

int grid_blocks(const AttnParams& p) {
  const int groups = p.nsplit * p.batch * p.hkv;
  return ((groups + 7) / 8) * 8 * p.row_groups;
}

}  // namespace

hipError_t launch_attn_bf16(const AttnParams& p, bool tree, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const dim3 grid(grid_blocks(p)), block(kWaves * 64);
  if (ev0) (void)hipEventRecord(ev0, s);
  if (p.d == 128) {
    if (tree) hipLaunchKernelGGL((attn_bf16_partial<128, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_bf16_partial<128, false>), grid, block, 0, s, p);
  } else {
    if (tree) hipLaunchKernelGGL((attn_bf16_partial<64, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_bf16_partial<64, false>), grid, block, 0, s, p);
  }
  hipError_t e = hipGetLastError();
  if (ev1) (void)hipEventRecord(ev1, s);
  return e;
}

}  // namespace glance
