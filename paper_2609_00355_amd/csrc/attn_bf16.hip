// Split-KV attention for the block draft and the ancestor-masked tree verify,
// bf16 in / fp32 accumulate, on gfx950 matrix cores.
//
// One workgroup owns one (sequence b, KV head g, context split s, row group).
// Its rows are the flattened (new row, query head of the group) pairs, so the
// K/V tile staged in LDS is shared by every query head of the GQA group and
// by every block/tree row: the context is read from HBM once per split.
//
// K/V tiles of 64 keys stream from HBM straight into LDS (global_load_lds,
// 16 bytes per lane, no register staging) through a ring of kStages buffers,
// so several tiles are in flight per workgroup while the current one is
// consumed.  Rows of the tile are stored unpadded with the 16-byte chunks of
// key k permuted by an XOR with swz(k), which keeps both the K-operand reads
// and the transposed V reads free of bank conflicts.  The loads are issued
// from inline assembly and waited for explicitly (s_waitcnt vmcnt), because
// the compiler, seeing a load into LDS in flight, would otherwise wait for
// all of them before every LDS read and drain the ring.
//
// Per tile each wave computes, for each of its 16-row tiles,
//   S^T[key][row] = K[key][:] . Q[row][:]        (v_mfma_f32_16x16x32_bf16, A = K, B = Q^T)
//   online softmax over the keys of each row    (exp2 with the scale folded in)
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

#include <type_traits>

namespace glance {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr float kNegInf = -__builtin_inff();
constexpr int kStages = 4;     // LDS ring depth: tiles in flight per workgroup
constexpr float kSlack = 8.f;  // lazy-rescale threshold (exp2 units)

template <int D>
struct Geom {
  static constexpr int kRowBytes = D * 2;                    // one key row, unpadded
  static constexpr int kChunks = D / 8;                      // 16-byte chunks per row
  static constexpr int kKeysPerInst = 64 / kChunks;          // rows filled by one wave load
  static constexpr int kTileBytes = kKeyTile * kRowBytes;    // one K (or V) tile
  static constexpr int kInstPerWave = kKeyTile / (kKeysPerInst * kBf16Waves);
};

// Chunk permutation of key row k (XOR, so a bijection on the chunks of a row).
// Lanes 0-7 of a K-operand read touch rows {0-3, 8-11} (+16 for lanes 8-15) at
// one chunk; lanes of a transposed V read touch 4 consecutive rows at two
// neighbouring chunks.  Both land on distinct 16-byte bank groups.
template <int D>
__device__ __forceinline__ int swz(int k) {
  if (D >= 128) return ((k & 3) << 1) | (((k >> 3) & 1) << 3) | ((k >> 4) & 1);
  return ((k & 3) << 1) | ((k >> 3) & 1);
}

// One 16-byte-per-lane load from global memory into LDS: lane i writes LDS
// bytes [lds_base + 16 i, +16).  M0 carries the wave-uniform LDS base; it is
// saved and restored around the load (the compiler owns M0), and one wait
// state separates the M0 write from the load that reads it.
__device__ __forceinline__ void dma16(const void* gptr, unsigned lds_base) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(gptr)
      : "memory");
}

// The same load with a wave-uniform 64-bit base in SGPRs and a 32-bit
// per-lane byte offset: no per-lane address arithmetic at issue.
__device__ __forceinline__ void dma16s(const void* sbase, unsigned voff, unsigned lds_base) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(voff), "s"(sbase)
      : "memory");
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Workgroup barrier for the DMA ring.  __syncthreads() carries a release fence,
// which would make every wave wait for all of its outstanding global->LDS
// loads (vmcnt(0)) and drain the ring.  Here each wave has already waited for
// the loads of the tile it is about to read (wait_vmcnt), so the barrier only
// has to order LDS: finish this wave's own LDS operations, then s_barrier.  The
// "memory" clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int D, bool TREE, int TPW>
__global__ __launch_bounds__(kBf16Waves * 64) void attn_bf16_partial(AttnParams p) {
  using G_ = Geom<D>;
  constexpr int KS = D / 32;  // k-steps of Q.K^T
  constexpr int DT = D / 16;  // d-tiles of P.V
  constexpr int RB = G_::kRowBytes;
  constexpr int CH = G_::kChunks;
  constexpr int IPW = G_::kInstPerWave;
  constexpr int LOADS_PER_TILE = 2 * IPW;  // K and V load instructions per wave per tile
  constexpr int kAhead = kStages - 1;  // tiles streaming behind the current one
  static_assert(IPW * G_::kKeysPerInst * kBf16Waves == kKeyTile, "tile load must divide evenly");

  __shared__ __attribute__((aligned(1024))) char sRing[kStages][2][G_::kTileBytes];
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
  // Full context tiles come first; the ragged last context tile and the
  // new-key tile (if any) need the mask.
  const int n_full = (k_end - k_begin) / kKeyTile;

  const __bf16* q = static_cast<const __bf16*>(p.q);
  const char* kc = static_cast<const char*>(p.k_ctx);
  const char* vc = static_cast<const char*>(p.v_ctx);
  const char* kn = static_cast<const char*>(p.k_new);
  const char* vn = static_cast<const char*>(p.v_new);

  // ---- the loads of tile t into ring stage st.  Wave w fills rows
  // [8w, 8w+8); lane i of a load writes LDS row base + i/CH, chunk slot i%CH,
  // which holds global chunk slot ^ swz(row).  Rows past the valid keys re-read
  // the last valid row: their scores are masked, so P = 0 and V is finite.
  // Lane offsets of the wave's shares within a full context tile (all 64 rows
  // valid, row stride RB), computed once; other tiles compute theirs at issue.
  unsigned full_off[LOADS_PER_TILE / 2];
#pragma unroll
  for (int i = 0; i < LOADS_PER_TILE / 2; ++i) {
    const int row = (wave * IPW + i) * G_::kKeysPerInst + lane / CH;
    full_off[i] = (unsigned)(row * RB + ((lane % CH) ^ swz<D>(row)) * 16);
  }
  auto issue = [&](int t) __attribute__((always_inline)) {
    // t is the same in every lane; say so, since the LDS base must sit in an SGPR
    // (M0) and the compiler's uniformity analysis can lose track of it in loops
    // whose bodies branch per lane.
    t = __builtin_amdgcn_readfirstlane(t);
    const unsigned lk = (unsigned)(size_t)(&sRing[t % kStages][0][0]);
    const unsigned lv = (unsigned)(size_t)(&sRing[t % kStages][1][0]);
    if (t < n_full) {
      // one tile base for all of the wave's shares: SGPR base + lane offsets
      const size_t off = (((size_t)b * p.hkv + g) * p.cap + k_begin + (size_t)t * kKeyTile) * RB;
#pragma unroll
      for (int i = 0; i < LOADS_PER_TILE / 2; ++i) {
        const unsigned lrow = (unsigned)((wave * IPW + i) * G_::kKeysPerInst * RB);
        dma16s(kc + off, full_off[i], lk + lrow);
        dma16s(vc + off, full_off[i], lv + lrow);
      }
      return;
    }
    const char* kb;
    const char* vb;
    size_t stride;
    int nvalid;
    if (t < n_ctx_tiles) {
      const int key0 = k_begin + t * kKeyTile;
      nvalid = min(kKeyTile, k_end - key0);
      const size_t off = (((size_t)b * p.hkv + g) * p.cap + key0) * RB;
      kb = kc + off;
      vb = vc + off;
      stride = RB;
    } else {
      nvalid = p.n;
      const size_t off = ((size_t)b * p.n * p.hkv + g) * RB;
      kb = kn + off;
      vb = vn + off;
      stride = (size_t)p.hkv * RB;
    }
    // The lane's offsets are recomputed from a laundered lane id each time:
    // hoisted out of the loop they would stay live across it and push the
    // kernel into spilling (whose reloads wait for every tile load in flight).
    int ln = lane;
    asm volatile("" : "+v"(ln));
#pragma unroll
    for (int i = 0; i < LOADS_PER_TILE / 2; ++i) {
      const int row0 = (wave * IPW + i) * G_::kKeysPerInst;
      const int row = row0 + ln / CH;
      const int src = row < nvalid ? row : nvalid - 1;
      const unsigned goff = (unsigned)src * (unsigned)stride + (unsigned)(((ln % CH) ^ swz<D>(row)) * 16);
      dma16(kb + goff, lk + row0 * RB);
      dma16(vb + goff, lv + row0 * RB);
    }
  };

  // ---- ancestor words of the packed tree, anc[i] = {i} u anc[parent(i)], by
  // pointer doubling in wave 0 (one load per node instead of a chain of
  // dependent loads): after r rounds lane i holds the nodes on its root path
  // from i up to (excluding) its 2^r-th ancestor up[i].
  // The query and parent loads below are issued from inline assembly, like
  // the tile loads, and waited for explicitly: the compiler counts only the
  // loads it can see, so its own wait before their first use would be
  // vmcnt(0) and would also wait for every tile load in flight.
  unsigned long long anc_word = 0;
  int up = -1;
  int par_raw = -1;
  const bool load_par = TREE && has_new && wave == 0 && lane < p.n;
  if (load_par)
    asm volatile("global_load_dword %0, %1, off" : "=v"(par_raw) : "v"(p.parents + (size_t)b * p.n + lane) : "memory");

  // ---- this wave's query rows, held as MFMA B operands for the whole split.
  const int n_row_tiles = (p.rows + 15) >> 4;
  const int tile0 = rg * p.tiles_per_group + wave * TPW;
  // Inactive tiles (past this row group or past the last row) compute on a
  // zero query and are not written; a wave with none skips the arithmetic.
  bool act[TPW];
  bf16x8 qf[TPW][KS];
  int node_of[TPW];
  bool wave_active = false;
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    act[j] = (wave * TPW + j < p.tiles_per_group) && (tile0 + j < n_row_tiles);
    wave_active = wave_active || act[j];
    const int row = (tile0 + j) * 16 + lr;
    node_of[j] = p.n;  // padding rows: treated as seeing every key
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[j][ks] = bf16x8{};
    if (act[j] && row < p.rows) {
      const int node = row / p.group;
      const int hl = row - node * p.group;
      node_of[j] = node;
      const __bf16* qp = q + (((size_t)b * p.n + node) * p.hq + (size_t)g * p.group + hl) * D + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        u32x4 raw;
        asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(raw) : "v"(qp + 32 * ks) : "memory");
        qf[j][ks] = as_bf16x8(raw);
      }
    }
  }

  // Then the first tiles start streaming.
#pragma unroll
  for (int t = 0; t < kAhead; ++t)
    if (t < n_tiles) issue(t);

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

  // ---- one tile, for each of this wave's 16-row tiles j:
  //   S^T[key][row] = K[key][:] . Q[row][:]   (A = K from LDS, B = Q^T)
  //   P = exp2(S c - m_run c)                  (online softmax, lazily rescaled)
  //   O^T[d][row] += V^T[d][key] . P^T[key][row]
  // The keys of a tile form two halves kk (keys 32 kk .. 32 kk + 31).  A lane
  // holds row lr and keys 32 kk + 8 lg + 4 sub + i of S^T (value sc[j][kk][sub][i]).
  //
  // The exponentials are computed against the running reference m_run before
  // the tile's maximum is known, so that they can be interleaved with matrix
  // work: those of half 0 with the Q.K MFMAs of half 1, those of half 1 with
  // the P.V MFMAs of half 0.  Lazy rescaling keeps the reference unless a
  // score exceeds it by more than 2^kSlack (exp2 units); in that rare case
  // (always on a split's first tile) the reference moves, O and l are
  // rescaled, and half 0 is scored again and exponentiated anew.
  //
  // Operand reads from LDS run kOpAhead operands ahead of their MFMAs, and
  // scheduling fences keep each step (one operand's MFMAs plus its share of
  // VALU work) in place, so the compiler neither regroups the reads (which
  // would expose their latency) nor separates the VALU work from the MFMAs.
  constexpr int NKO = 4 * KS;        // K operands per tile: (kk, ks, sub)
  constexpr int NVO = 2 * DT;        // V operands per tile: (kk, dt)
  constexpr int kOpAhead = 2;
  constexpr int NVAL = TPW * 8;      // scores per lane in one half
  static_assert(NKO / 2 == 2 * KS && NVO / 2 == DT, "operand counts");

  auto tile = [&](auto masked_tag, int t) __attribute__((always_inline)) {
    constexpr bool masked = decltype(masked_tag)::value;
    const char* Kt = sRing[t % kStages][0];
    const char* Vt = sRing[t % kStages][1];
    const bool is_new = (t == n_ctx_tiles);
    const int nvalid = is_new ? p.n : min(kKeyTile, k_end - (k_begin + t * kKeyTile));

    auto load_k = [&](int idx) __attribute__((always_inline)) {
      const int kk = idx / (2 * KS), ks = (idx / 2) % KS, sub = idx % 2;
      const int krow = 32 * kk + 8 * (lr >> 2) + 4 * sub + (lr & 3);
      return as_bf16x8(*reinterpret_cast<const u32x4*>(Kt + krow * RB + ((4 * ks + lg) ^ swz<D>(krow)) * 16));
    };
    // V^T operand of (kk, dt): two transposed 8-byte reads, rows vrow and vrow + 4.
    // ds_read_b64_tr_b16: in each 16-lane group, lane jl reads row key0 + (jl>>2),
    // columns d0 + 4*(jl&3) .. +3, and receives V[key0 + i][d0 + jl] for i = 0..3.
    auto load_v = [&](int idx) __attribute__((always_inline)) {
      const int kk = idx / DT, dt = idx % DT;
      const int vrow = 32 * kk + 8 * lg + (lr >> 2);
      const int chunk = 2 * dt + ((lane & 3) >> 1);
      const int half = (lane & 1) * 8;
      const char* va_lo = Vt + vrow * RB + (chunk ^ swz<D>(vrow)) * 16 + half;
      const char* va_hi = Vt + (vrow + 4) * RB + (chunk ^ swz<D>(vrow + 4)) * 16 + half;
      const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(va_lo));
      const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(va_hi));
      // whole-vector reinterpretation: element-wise bf16 inserts of the 16-bit
      // lanes were miscompiled (every element became lo[0])
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };

    f32x4 sc[TPW][2][2];
    bf16x8 kr[kOpAhead + 1];
    auto qk_step = [&](int idx) __attribute__((always_inline)) {
      if (idx + kOpAhead < NKO) kr[(idx + kOpAhead) % (kOpAhead + 1)] = load_k(idx + kOpAhead);
      const int kk = idx / (2 * KS), ks = (idx / 2) % KS, sub = idx % 2;
#pragma unroll
      for (int j = 0; j < TPW; ++j)
        sc[j][kk][sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[idx % (kOpAhead + 1)], qf[j][ks],
                                                                ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sc[j][kk][sub],
                                                                0, 0, 0);
    };
    // Q.K^T of half kk alone (used again by the rescale path)
    auto qk_half = [&](int kk) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < kOpAhead; ++i) kr[(kk * 2 * KS + i) % (kOpAhead + 1)] = load_k(kk * 2 * KS + i);
#pragma unroll
      for (int n = 0; n < 2 * KS; ++n) {
        const int idx = kk * 2 * KS + n;
        if (n + kOpAhead < 2 * KS) kr[(idx + kOpAhead) % (kOpAhead + 1)] = load_k(idx + kOpAhead);
        const int ks = n / 2, sub = n % 2;
#pragma unroll
        for (int j = 0; j < TPW; ++j)
          sc[j][kk][sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              kr[idx % (kOpAhead + 1)], qf[j][ks], ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sc[j][kk][sub], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    auto mask_half = [&](int kk) __attribute__((always_inline)) {
      if (!masked) return;
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        unsigned long long anc = ~0ull;
        if (TREE && is_new && node_of[j] < p.n) anc = sAnc[node_of[j]];
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = 32 * kk + 8 * lg + 4 * sub + i;
            bool vis = key < nvalid;
            if (TREE && is_new) vis = vis && ((anc >> key) & 1ull);
            if (!vis) sc[j][kk][sub][i] = kNegInf;
          }
      }
    };

    float mx[TPW], ls[TPW], neg[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      mx[j] = kNegInf;
      ls[j] = 0.f;
      neg[j] = -m_run[j] * c;
    }
    // score n of half kk -> probability (argument <= kSlack unless the
    // reference moves; v_exp_f32 flushes the far tail to 0)
    auto exp_item = [&](int kk, int n, bool track_max) __attribute__((always_inline)) {
      const int j = n / 8, sub = (n / 4) % 2, i = n % 4;
      const float v = sc[j][kk][sub][i];
      if (track_max) mx[j] = fmaxf(mx[j], v);
      float e = __builtin_amdgcn_exp2f(fmaf(v, c, neg[j]));
      // pin the exponential here: the rescale path recomputes half 0, so the
      // compiler would otherwise sink these below the check, out of the MFMA stream
      asm volatile("" : "+v"(e));
      sc[j][kk][sub][i] = e;
    };

    // Phase 1: Q.K^T of half 0 (matrix work only).
#pragma unroll
    for (int i = 0; i < kOpAhead; ++i) kr[i] = load_k(i);
#pragma unroll
    for (int idx = 0; idx < NKO / 2; ++idx) {
      qk_step(idx);
      __builtin_amdgcn_sched_barrier(0);
    }
    // Phase 2: Q.K^T of half 1, with the exponentials of half 0.
    mask_half(0);
#pragma unroll
    for (int n = 0; n < NKO / 2; ++n) {
      qk_step(NKO / 2 + n);
#pragma unroll
      for (int m = n * NVAL / (NKO / 2); m < (n + 1) * NVAL / (NKO / 2); ++m) exp_item(0, m, true);
      __builtin_amdgcn_sched_barrier(0);
    }
    // The first V operands stream in while the maximum is checked.
    bf16x8 vr[kOpAhead + 1];
#pragma unroll
    for (int i = 0; i < kOpAhead; ++i) vr[i] = load_v(i);
    mask_half(1);
#pragma unroll
    for (int j = 0; j < TPW; ++j)
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int i = 0; i < 4; ++i) mx[j] = fmaxf(mx[j], sc[j][1][sub][i]);
    // Each lane tests its own maximum: no lane above the reference means no row is.
    bool move = false;
#pragma unroll
    for (int j = 0; j < TPW; ++j) move = move | (mx[j] * c > m_run[j] * c + kSlack) | (m_run[j] == kNegInf);
    if (__builtin_amdgcn_ballot_w64(move)) {
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        float m = mx[j];
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        const float m_new = fmaxf(m_run[j], m);
        const float m_use = (m_new == kNegInf) ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f((m_run[j] - m_use) * c);
        m_run[j] = m_use;
        l_run[j] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[j][dt] *= alpha;
        neg[j] = -m_use * c;
      }
      // half 0 was exponentiated against the old reference: score it again
      qk_half(0);
      mask_half(0);
#pragma unroll
      for (int m = 0; m < NVAL; ++m) exp_item(0, m, false);
    }
    __builtin_amdgcn_sched_barrier(0);

    // Phase 3: P.V of half 0, with the exponentials of half 1.
    bf16x8 pb[TPW];
    // Probabilities of half kk as the bf16 B operand of P.V; the row sum l
    // is taken from these same bf16 values (two per v_dot2c_f32_bf16), so
    // numerator and denominator use identical weights.
    auto to_pb = [&](int kk) __attribute__((always_inline)) {
      typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
      const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pb[j][i] = (__bf16)sc[j][kk][0][i];
          pb[j][4 + i] = (__bf16)sc[j][kk][1][i];
        }
        ls[j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[j], pb[j], 0, 1), ones, ls[j], false);
        ls[j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[j], pb[j], 2, 3), ones, ls[j], false);
        ls[j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[j], pb[j], 4, 5), ones, ls[j], false);
        ls[j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[j], pb[j], 6, 7), ones, ls[j], false);
      }
    };
    auto pv_step = [&](int idx) __attribute__((always_inline)) {
      if (idx + kOpAhead < NVO) vr[(idx + kOpAhead) % (kOpAhead + 1)] = load_v(idx + kOpAhead);
      const int dt = idx % DT;
#pragma unroll
      for (int j = 0; j < TPW; ++j)
        o[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vr[idx % (kOpAhead + 1)], pb[j], o[j][dt], 0, 0, 0);
    };
    to_pb(0);
#pragma unroll
    for (int n = 0; n < DT; ++n) {
      pv_step(n);
#pragma unroll
      for (int m = n * NVAL / DT; m < (n + 1) * NVAL / DT; ++m) exp_item(1, m, false);
      __builtin_amdgcn_sched_barrier(0);
    }
    // Phase 4: P.V of half 1.
    to_pb(1);
#pragma unroll
    for (int n = 0; n < DT; ++n) {
      pv_step(DT + n);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < TPW; ++j) l_run[j] += ls[j];
  };

  // Queries and parents were issued before the tile loads, so they have
  // landed once no more than the tile loads are outstanding.  The query
  // registers pass through the wait so that no use moves above it.
  if (n_tiles >= kAhead) {
#pragma unroll
    for (int j = 0; j < TPW; ++j)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        u32x4 raw = __builtin_bit_cast(u32x4, qf[j][ks]);
        if (j == 0 && ks == 0)
          asm volatile("s_waitcnt vmcnt(%1)" : "+v"(raw) : "n"(kAhead * LOADS_PER_TILE) : "memory");
        else
          asm volatile("" : "+v"(raw));
        qf[j][ks] = as_bf16x8(raw);
      }
  } else {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  if (load_par) {
    asm volatile("" : "+v"(par_raw));
    up = (par_raw >= 0 && par_raw < lane) ? par_raw : -1;
    anc_word = 1ull << lane;
  }

  if (TREE && has_new && wave == 0) {
#pragma unroll
    for (int r = 0; r < 6; ++r) {
      const int src = up < 0 ? lane : up;
      const unsigned lo = __shfl((unsigned)anc_word, src);
      const unsigned hi = __shfl((unsigned)(anc_word >> 32), src);
      const int up2 = __shfl(up, src);
      if (up >= 0) {
        anc_word |= ((unsigned long long)hi << 32) | lo;
        up = up2;
      }
    }
    if (lane < p.n) sAnc[lane] = anc_word;  // read after the loop's barriers
  }

  // Barrier j: every wave's loads of tile j have landed (each wave waits for
  // its own share first), and the ring stage that tile j + kAhead will use is
  // free, so the loads of that tile are issued right after it.  (Issuing them
  // from inside the tile, between the matrix phases, bought no speed and gave
  // intermittently wrong tree-verify rows, so they stay here.)
  auto barrier_step = [&](int j) __attribute__((always_inline)) {
    if (j < n_tiles) {
      if (j + kAhead - 1 < n_tiles) wait_vmcnt<(kAhead - 1) * LOADS_PER_TILE>();
      else wait_vmcnt<0>();
    }
    lds_barrier();
    if (j + kAhead < n_tiles) issue(j + kAhead);
  };

  // All waves in step: tile t is consumed between barriers t and t + 1 while
  // kAhead tiles stream behind it.  Full context tiles run first, through a
  // loop whose body carries no mask; the ragged last context tile and the
  // new-key tile follow with it.
  {
    int t = 0;
    for (; t < n_full; ++t) {
      barrier_step(t);
      if (wave_active) tile(std::false_type{}, t);
    }
    for (; t < n_tiles; ++t) {
      barrier_step(t);
      if (wave_active) tile(std::true_type{}, t);
    }
  }

  // ---- partial results of this split: O unnormalised, (max * c, sum).
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    if (!act[j]) continue;
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

template <int D, bool TREE>
void launch_d(const AttnParams& p, hipStream_t s) {
  const dim3 grid(grid_blocks(p)), block(kBf16Waves * 64);
  if (p.tiles_per_wave == 2) hipLaunchKernelGGL((attn_bf16_partial<D, TREE, 2>), grid, block, 0, s, p);
  else hipLaunchKernelGGL((attn_bf16_partial<D, TREE, 1>), grid, block, 0, s, p);
}

}  // namespace

hipError_t launch_attn_bf16(const AttnParams& p, bool tree, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (ev0) (void)hipEventRecord(ev0, s);
  if (p.d == 128) {
    if (tree) launch_d<128, true>(p, s);
    else launch_d<128, false>(p, s);
  } else {
    if (tree) launch_d<64, true>(p, s);
    else launch_d<64, false>(p, s);
  }
  hipError_t e = hipGetLastError();
  if (ev1) (void)hipEventRecord(ev1, s);
  return e;
}

}  // namespace glance
