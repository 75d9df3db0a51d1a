// Split-KV attention for the block draft and the ancestor-masked tree verify,
// bf16 in / fp32 accumulate, on gfx950 matrix cores.
//
// Work items.  The rows of one (sequence b, KV head g) problem are the
// flattened (new row, query head of the GQA group) pairs, so one K/V tile in
// LDS serves every query head of the group and every block or tree row.  The
// rows form row groups of up to seven 32-row tiles; the keys of a sequence
// (its context tiles of 64 keys, then one tile holding the block or tree keys)
// are cut into pieces.  A workgroup owns one (piece, row group).  The pieces
// are planned on the device from ctx_lens, the same way by every workgroup:
// each sequence of len_b tiles gets n_b = ceil(len_b / T) pieces of nearly
// equal size, with T the smallest size for which all pieces fit the launched
// slots; so a ragged batch gets pieces of equal cost rather than equal key
// ranges, and no slot is spent on a sequence's padding.
//
// Waves.  Waves 0 .. tiles-1 compute one 32-row tile each.  The waves
// without rows (one to four of them issue) stream K/V tiles from HBM straight
// into LDS (global_load_lds, 16 bytes per lane, no register staging), each
// its share of every tile, through rings of four K stages and four V stages;
// one LDS barrier per tile orders the loads and the reads (the ring's rule
// is stated at ring_wait).
//
// Per tile a computing wave runs, for its 32 rows and the tile's 64 keys,
//   S^T[key][row] = K[key][:] . Q[row][:]           (v_mfma_f32_32x32x16_bf16, A = K, B = Q^T)
//   P = exp2(S c - m c)                              (online softmax, lazily rescaled)
//   O^T[d][row] += V^T[d][key] . P^T[key][row]     (A = V^T by ds_read_b64_tr_b16, B = P^T)
// as a matrix phase (Q.K^T of tile t with P.V of tile t-1) and a vector phase
// (the softmax of tile t); the two waves that share a SIMD overlap one's
// matrix phase with the other's vector phase.  The
// MFMA result layout of S^T (lane l: row l%32, keys 8j + 4(l/32) + i) is used
// directly as the B operand of P.V by ordering the keys of each 16-key k-step
// accordingly (no shuffles), and the row of a lane never changes, so the
// running max and sum are per lane (lanes l and l+32 share a row).
//
// Merge.  A piece that is its sequence's only one writes the output and LSE.
// Otherwise each piece writes its unnormalised output (in the MFMA register
// layout, one float4 per lane per store) and (max, sum) per row to the
// workspace, and attn_merge.hip combines the pieces in a second, fully
// parallel pass; the first piece of each sequence records the sequence's
// piece count and first slot for it.
#include "glance_internal.h"

namespace glance {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(4))) _Float16 f16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) char lds_char;

constexpr float kNegInf = -__builtin_inff();
constexpr int kStages = 4;          // LDS ring depth (tiles)
constexpr float kSumLimit = 256.f;  // per-lane probability sum that forces a rescale
constexpr float kLn2 = 0.6931471805599453f;
#ifndef GLANCE_AHEAD
#define GLANCE_AHEAD 2
#endif
#ifndef GLANCE_XPRIO
#define GLANCE_XPRIO 1  // raised wave priority during the matrix phase
#endif
constexpr int kOperandsAhead = GLANCE_AHEAD;  // LDS operand reads issued ahead of their MFMA

// Key-tile geometry for head dimension D (bf16 rows, unpadded).
template <int D>
struct Geo {
  static constexpr int RB = 2 * D;      // bytes per key row
  static constexpr int CH = D / 8;      // 16-byte chunks per row
  static constexpr int TB = 64 * RB;    // bytes of one K (or V) tile
  static constexpr int KS = D / 16;     // k-steps of Q.K^T (16 dims each)
  static constexpr int DB = D / 32;     // 32-dim blocks of P.V
  static constexpr int RPL = 1024 / RB; // key rows per 1 KB load instruction
  static constexpr int NB = 64 / RPL;   // load instructions per K (or V) tile
  static constexpr int OV = D / 2;      // fp32 output values per lane (32 rows x D / 64)
};

// Chunk c of key row r sits at chunk c ^ swz(r) of the row's LDS slot.  The
// LDS serves 64 banks of 4 bytes; a K-operand read (16 bytes per lane) covers
// 16 consecutive rows at one chunk per 16 lanes, and a transposed V read
// covers 4 consecutive rows x 2 chunks per 16 lanes.  swz is a bijection on
// the 16-byte bank groups over every aligned run of 16 rows (bits 0-3), and
// over every aligned run of 4 rows both bits 1-2 and bits 2-3 run through all
// four values, so both reads are free of bank conflicts (measured against
// simpler permutations).  For D = 64 (8 chunks per row) only bits 0-2 apply.
template <int D>
__device__ __forceinline__ int swz(int r) {
  const int t = 8 * ((r >> 1) & 1) + 4 * (r & 1) + 2 * (((r >> 1) ^ r) & 1) + ((r >> 2) & 1);
  const int s = t ^ (((r >> 3) & 1) << 1);
  return D >= 128 ? s : (s & 7);
}

// One 16-byte-per-lane load from global memory into LDS: lane i writes LDS
// bytes [lds + 16 i, +16) with data from sbase + voff.  M0 carries the LDS
// address; it is saved and restored around the load (the compiler owns M0).
__device__ __forceinline__ void dma16(const void* sbase, unsigned voff, unsigned lds) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(voff), "s"(sbase)
      : "memory");
}

// s_waitcnt vmcnt(N), other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// Barrier that orders LDS only: this wave's LDS operations finish, then
// s_barrier.  (__syncthreads() also waits for every outstanding global load,
// which would drain the ring.)
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, __shfl_xor(v, off));
  return v;
}

__device__ __forceinline__ int clamp_ctx(int ctx, int cap) { return ctx < 0 ? 0 : (ctx > cap ? cap : ctx); }
// tiles of a sequence: its context tiles, then the tile of new keys
__device__ __forceinline__ int seq_tiles(int ctx) { return (ctx + 63) / 64 + 1; }

struct Piece {
  int b;        // sequence
  int first;    // piece slot of the sequence's first piece (within the KV head)
  int count;    // pieces of the sequence
  int index;    // this piece's index among them
  int t_begin;  // first tile (of the sequence's tile list)
  int n_tiles;  // tiles of the piece, >= 1
  int ctx;      // context keys of the sequence
};

// The piece plan (identical in every wave of every workgroup): T is the
// smallest piece size, at least min_tiles, with sum_b ceil(len_b / T) <=
// slots; piece slot ps then names piece ps - first_b of the sequence b with
// first_b <= ps < first_b + n_b.  Returns false if the slot is unused.  The
// lengths are read once (sequences lane + 64 k, k < kPlanCache, held in
// registers; larger batches re-read the rest), since every memory round trip
// here delays the first tile load.
constexpr int kPlanCache = 4;
__device__ bool find_piece(const AttnParams& p, int ps, int lane, Piece& out) {
  int len_c[kPlanCache], ctx_c[kPlanCache];
#pragma unroll
  for (int k = 0; k < kPlanCache; ++k) {
    const int b = lane + 64 * k;
    ctx_c[k] = b < p.batch ? clamp_ctx(p.ctx_lens[b], p.cap) : 0;
    len_c[k] = b < p.batch ? seq_tiles(ctx_c[k]) : 0;
  }
  auto len_of = [&](int k, int b) __attribute__((always_inline)) {
    return k < kPlanCache ? len_c[k] : (b < p.batch ? seq_tiles(clamp_ctx(p.ctx_lens[b], p.cap)) : 0);
  };
  int total = 0, longest = 0;
  for (int b0 = 0, k = 0; b0 < p.batch; b0 += 64, ++k) {
    const int len = len_of(k, b0 + lane);
    total += len;
    longest = max(longest, len);
  }
  total = wave_sum(total);
  longest = wave_max(longest);
  const int slots = p.slots_per_g;
  auto count = [&](int T) __attribute__((always_inline)) {
    int cnt = 0;
    for (int b0 = 0, k = 0; b0 < p.batch; b0 += 64, ++k) cnt += (len_of(k, b0 + lane) + T - 1) / T;
    return wave_sum(cnt);
  };
  int lo = max(p.min_tiles, (total + slots - 1) / slots);
  int hi = max(lo, longest);  // with T = longest every sequence is one piece; slots >= batch
  if (count(lo) <= slots) hi = lo;  // exact for equal lengths
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (count(mid) <= slots) hi = mid;
    else lo = mid + 1;
  }
  const int T = __builtin_amdgcn_readfirstlane(lo);
  int base = 0;
  for (int b0 = 0, k = 0; b0 < p.batch; b0 += 64, ++k) {
    const int b = b0 + lane;
    const int ctx = k < kPlanCache ? ctx_c[k] : (b < p.batch ? clamp_ctx(p.ctx_lens[b], p.cap) : 0);
    const int len = b < p.batch ? seq_tiles(ctx) : 0;
    const int nb = (len + T - 1) / T;
    int incl = nb;  // inclusive prefix sum over the lanes
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    incl += base;
    const int excl = incl - nb;
    const unsigned long long hit = __ballot(b < p.batch && excl <= ps && ps < incl);
    if (hit) {
      const int src = __ffsll((long long)hit) - 1;
      out.b = b0 + src;
      out.first = __shfl(excl, src);
      out.count = __shfl(nb, src);
      out.ctx = __shfl(ctx, src);
      const int slen = __shfl(len, src);
      out.index = ps - out.first;
      out.t_begin = out.index * slen / out.count;
      out.n_tiles = (out.index + 1) * slen / out.count - out.t_begin;
      out.b = __builtin_amdgcn_readfirstlane(out.b);
      out.first = __builtin_amdgcn_readfirstlane(out.first);
      out.count = __builtin_amdgcn_readfirstlane(out.count);
      out.ctx = __builtin_amdgcn_readfirstlane(out.ctx);
      out.index = __builtin_amdgcn_readfirstlane(out.index);
      out.t_begin = __builtin_amdgcn_readfirstlane(out.t_begin);
      out.n_tiles = __builtin_amdgcn_readfirstlane(out.n_tiles);
      return true;
    }
    base = __shfl(incl, 63);
  }
  return false;
}

template <int D, bool TREE>
__global__ __launch_bounds__(512) void attn_bf16(AttnParams p) {
  using G_ = Geo<D>;
  constexpr int RB = G_::RB, CH = G_::CH, TB = G_::TB, KS = G_::KS, DB = G_::DB;
  constexpr int RPL = G_::RPL, NB = G_::NB, OV = G_::OV;

  __shared__ __attribute__((aligned(1024))) char sK[kStages * TB];
  __shared__ __attribute__((aligned(1024))) char sV[kStages * TB];
  __shared__ unsigned long long sAnc[64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  // ---- work item.  Blocks 8 (rg j + r) + x hold slot 8 j + x, row group r:
  // the row groups of one piece sit on one XCD (block index mod 8), so their
  // repeated K/V reads hit that XCD's L2.
  const int L = blockIdx.x;
  const int q8 = L >> 3;
  const int rgi = q8 % p.row_groups;
  const int slot = (q8 / p.row_groups) * 8 + (L & 7);
  if (slot >= p.slots_per_g * p.hkv) return;
  const int g = slot / p.slots_per_g;
  Piece pc;
  if (!find_piece(p, slot - g * p.slots_per_g, lane, pc)) return;
  const int b = pc.b;
  const int ctx = pc.ctx;
  const int ct = (ctx + 63) / 64;  // context tiles; tile ct holds the new keys
  const int n_tiles = pc.n_tiles;
  const int tb = pc.t_begin;
  const bool has_new = tb + n_tiles - 1 == ct;
  const bool split = pc.count > 1;
  if (pc.index == 0 && g == 0 && rgi == 0 && threadIdx.x == 0)
    p.plan[b] = make_int2(pc.count, pc.first);  // for the merge pass

  // =========================== K/V streaming ===========================
  // A DMA instruction holds its wave until the memory pipeline takes it,
  // hundreds of cycles when HBM is busy.  With at most four computing waves,
  // waves 4-7 (which have no rows) issue everything and the computing waves
  // none; with five to seven, every wave issues an equal share (one or two
  // waves without rows could not issue a whole tile's loads in the time the
  // computing waves take for it).
  const char* kc = static_cast<const char*>(p.k_ctx);
  const char* vc = static_cast<const char*>(p.v_ctx);
  const char* kn = static_cast<const char*>(p.k_new);
  const char* vn = static_cast<const char*>(p.v_new);
  // This wave's loads of a K (or V) tile: r = first + stride i, i < per_side.
  constexpr int kMaxLoads = NB / 4;
  int first, stride, per_side;
  if (p.tiles_rg <= 4) {
    first = wave - 4;
    stride = 4;
    per_side = wave >= 4 ? NB / 4 : 0;
  } else {
    first = wave;
    stride = 8;
    per_side = NB / 8;
  }
  // Load r (0 <= r < NB) of a tile fills LDS rows r RPL .. r RPL + RPL - 1;
  // lane i writes row r RPL + i / CH, chunk slot i % CH, which holds the
  // row's chunk slot ^ swz(row).  The lane's row and its byte offset within
  // a full context tile (row stride RB) are computed once per load slot.
  int lrow[kMaxLoads];
  unsigned lchunk[kMaxLoads];
#pragma unroll
  for (int i = 0; i < kMaxLoads; ++i) {
    lrow[i] = (first + stride * i) * RPL + lane / CH;
    lchunk[i] = (unsigned)(((lane % CH) ^ swz<D>(lrow[i])) * 16);
  }
  auto issue = [&](int t, bool v_side) __attribute__((always_inline)) {
    const char* gfull = v_side ? vc : kc;
    const unsigned lds = (unsigned)(size_t)(v_side ? sV : sK) + (unsigned)(t % kStages) * TB + first * 1024;
    const int j = tb + t;
    if (j < ct && 64 * j + 64 <= ctx) {  // full context tile: SGPR base + fixed lane offsets
      const char* base = gfull + (((size_t)b * p.hkv + g) * p.cap + 64 * (size_t)j) * RB;
#pragma unroll
      for (int i = 0; i < kMaxLoads; ++i)
        if (i < per_side) dma16(base, (unsigned)(lrow[i] * RB) + lchunk[i], lds + stride * i * 1024);
      return;
    }
    // ragged context tile or the new keys: rows past the valid ones re-read
    // the last valid row (their scores are masked, so P = 0 and V is finite)
    const char* base;
    unsigned rstride;
    int nvalid;
    if (j < ct) {
      base = gfull + (((size_t)b * p.hkv + g) * p.cap + 64 * (size_t)j) * RB;
      rstride = RB;
      nvalid = ctx - 64 * j;
    } else {
      base = (v_side ? vn : kn) + ((size_t)b * p.n * p.hkv + g) * RB;
      rstride = (unsigned)p.hkv * RB;
      nvalid = p.n;
    }
#pragma unroll
    for (int i = 0; i < kMaxLoads; ++i) {
      if (i < per_side) {
        const int src = lrow[i] < nvalid ? lrow[i] : nvalid - 1;
        dma16(base, (unsigned)src * rstride + lchunk[i], lds + stride * i * 1024);
      }
    }
  };
  // Ring rule.  Tile t is read by the computing waves' matrix phases: K(t) in
  // X_t, V(t) in X_{t+1} (see the schedule below); X_{t-1} ends before barrier
  // t in every wave.  So right after barrier t the stages of K(t - 1) and
  // V(t - 2) are free, and before barrier t + 1 each wave issues its share of
  // K(t + 3) and V(t + 2) into them (group t; the prologue issues groups -3,
  // -2, -1: K(0), then K(1) V(0), then K(2) V(1)).  Barrier t needs K(t) and
  // V(t - 1), both of group t - 3, so before it each wave waits until at most
  // its groups t - 2 and t - 1 are in flight (vmcnt counts this wave's loads,
  // in issue order): 2 per_side loads a group, so 4 per_side.  Every wave
  // issues its share of every group: a share left out leaves stale rows in
  // the stage, which the computing waves then read as tile data.
  auto ring_issue = [&](int t) __attribute__((always_inline)) {
    if (per_side == 0) return;
    if (t + 3 < n_tiles) issue(t + 3, false);
    if (t + 2 < n_tiles) issue(t + 2, true);
  };
  auto ring_prologue = [&]() __attribute__((always_inline)) {
    if (per_side == 0) return;
    issue(0, false);                    // group -3: K(0)
    if (n_tiles > 1) issue(1, false);   // group -2: K(1), V(0)
    issue(0, true);
    if (n_tiles > 2) issue(2, false);   // group -1: K(2), V(1)
    if (n_tiles > 1) issue(1, true);
  };
  auto ring_wait = [&](int t) __attribute__((always_inline)) {
    if (per_side == 0) return;
    if (t + 2 >= n_tiles) wait_vmcnt<0>();
    else if (per_side == NB / 4) wait_vmcnt<NB>();  // 4 per_side
    else wait_vmcnt<NB / 2>();                      // per_side = NB / 8
  };

  if (wave >= p.tiles_rg) {
    // a wave without rows: streams its share of the tiles and keeps the
    // barrier count
    ring_prologue();
    for (int t = 0; t < n_tiles; ++t) {
      ring_wait(t);
      lds_barrier();
      ring_issue(t);
    }
    return;
  }

  // =========================== computing waves ===========================
  const int h = lane >> 5;    // lane half: keys 4h.. of each 8-key group, dims 8h.. of each k-step
  const int r32 = lane & 31;  // the lane's row within the wave's tile
  const int row = 32 * (rgi * p.tiles_rg + wave) + r32;  // row of the (b, g) problem
  const bool row_ok = row < p.rows;
  const int node = row_ok ? row / p.group : p.n;
  const int hl = row_ok ? row - node * p.group : 0;
  const size_t out_row = ((size_t)b * p.n + node) * p.hq + (size_t)g * p.group + hl;

  // This wave's share of the first three ring groups, then the query of the
  // lane's row (dims 16 ks + 8 h .. +7: the B operands of Q.K^T) and (wave 0,
  // tree) the parents, all in flight together.  The query and parents are
  // ordinary loads issued after the tile loads: a wait the compiler places
  // for them (it counts only the loads it sees) also covers the older tile
  // loads, which completes more than it needs but never less.
  ring_prologue();
  bf16x8 qf[KS];
  {
    const __bf16* qp = static_cast<const __bf16*>(p.q) + out_row * D + 8 * h;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = row_ok ? *reinterpret_cast<const bf16x8*>(qp + 16 * ks) : bf16x8{};
  }
  const bool tree_words = TREE && has_new && wave == 0;
  int par = -1;
  if (tree_words && lane < p.n) par = p.parents[(size_t)b * p.n + lane];
  ring_wait(0);
  // ancestor words of the packed tree, anc[i] = {i} u anc[parent(i)], by
  // pointer doubling in wave 0: after r rounds lane i holds its root path
  // from i up to (excluding) its 2^r-th ancestor up[i]
  if (tree_words) {
    int up = (par >= 0 && par < lane) ? par : -1;
    unsigned long long anc = 1ull << lane;
#pragma unroll
    for (int r = 0; r < 6; ++r) {
      const int src = up < 0 ? lane : up;
      const unsigned lo = __shfl((unsigned)anc, src);
      const unsigned hi = __shfl((unsigned)(anc >> 32), src);
      const int up2 = __shfl(up, src);
      if (up >= 0) {
        anc |= ((unsigned long long)hi << 32) | lo;
        up = up2;
      }
    }
    if (lane < p.n) sAnc[lane] = anc;  // read after the tile barriers
  }

  // LDS read bases.  K operand (kb, ks): row 32 kb + r32, chunk 2 ks + h.
  // V^T operand (kb, s, db): two transposed reads of rows
  // 32 kb + 16 s + 4 (gr >> 1) + (jl >> 2) (+ 8), dims 32 db + 16 (gr & 1) +
  // 4 (jl & 3), gr = lane >> 4, jl = lane & 15: lane l receives
  // V[key][32 db + l % 32] for the keys 32 kb + 16 s + 4 h + 0..3 (+ 8), the
  // key order of the score layout.  The swizzle depends on the row modulo 16
  // only, so all but a per-lane base is an immediate offset (stage, kb, s),
  // and the tile loop is unrolled over the four stages.
  const lds_char* kbase[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) kbase[ks] = (const lds_char*)sK + r32 * RB + (((2 * ks + h) ^ swz<D>(r32)) * 16);
  const lds_char* vbase[DB][2];
  {
    const int gr = lane >> 4, jl = lane & 15;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int hi = 0; hi < 2; ++hi) {
        const int row = 8 * hi + 4 * (gr >> 1) + (jl >> 2);
        const int chunk = 4 * db + 2 * (gr & 1) + ((jl & 3) >> 1);
        vbase[db][hi] = (const lds_char*)sV + row * RB + ((chunk ^ swz<D>(row)) * 16) + 8 * (jl & 1);
      }
  }

  f32x16 S[2];  // scores of the current tile [key block]
  f32x16 O[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) O[db] = f32x16{};
  u32x4 Pw[2][2];  // probabilities as bf16 pairs [key block][16-key k-step]
  float m_run = kNegInf, l_run = 0.f, nmc = 0.f;
  const float c = p.scale_log2;

  auto load_k = [&](int ks, int kb, int st) __attribute__((always_inline)) {
    return __builtin_bit_cast(bf16x8, *(const lds_u32x4*)(kbase[ks] + st * TB + kb * 32 * RB));
  };
  auto load_v = [&](int u, int db, int st) __attribute__((always_inline)) {
    const int off = st * TB + (32 * (u >> 1) + 16 * (u & 1)) * RB;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbase[db][0] + off));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbase[db][1] + off));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };

  // scores (kb, j, i = 0..3) -> probabilities into Pw and their sum (from the
  // same bf16 values that P.V uses, so numerator and denominator match)
  auto soft_group = [&](int kb, int j, float& lsum) __attribute__((always_inline)) {
    const float e0 = __builtin_amdgcn_exp2f(fmaf(S[kb][4 * j + 0], c, nmc));
    const float e1 = __builtin_amdgcn_exp2f(fmaf(S[kb][4 * j + 1], c, nmc));
    const float e2 = __builtin_amdgcn_exp2f(fmaf(S[kb][4 * j + 2], c, nmc));
    const float e3 = __builtin_amdgcn_exp2f(fmaf(S[kb][4 * j + 3], c, nmc));
    const bf16x2 w0 = {(__bf16)e0, (__bf16)e1};
    const bf16x2 w1 = {(__bf16)e2, (__bf16)e3};
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    lsum = __builtin_amdgcn_fdot2_f32_bf16(w0, ones, lsum, false);
    lsum = __builtin_amdgcn_fdot2_f32_bf16(w1, ones, lsum, false);
    Pw[kb][j >> 1][2 * (j & 1)] = __builtin_bit_cast(unsigned, w0);
    Pw[kb][j >> 1][2 * (j & 1) + 1] = __builtin_bit_cast(unsigned, w1);
  };

  // Softmax of tile t (phase Y): mask a ragged or new-key tile (key
  // 32 kb + 8 j + 4 h + i is visible if it is valid and, in the tree, an
  // ancestor-or-self of the row's node), then the probabilities against the
  // running reference.  The reference moves to the row maximum when a lane's
  // probability sum passes kSumLimit (a score more than log2(kSumLimit) / c
  // above the reference) or there is no reference yet: O and l are rescaled
  // and the tile's probabilities redone.
  auto yphase = [&](int t) __attribute__((always_inline)) {
    const int j = tb + t;
    const bool is_new = j == ct;
    const int nvalid = is_new ? p.n : min(64, ctx - 64 * j);
    if (is_new || nvalid < 64) {
      unsigned long long anc = ~0ull;
      if (TREE && is_new && node < p.n) anc = sAnc[node];
      anc >>= 4 * h;
      const int lim = nvalid - 4 * h;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int k0 = 32 * kb + 8 * jj + i;  // key - 4 h
            bool vis = k0 < lim;
            if (TREE && is_new) vis = vis && ((anc >> k0) & 1ull);
            if (!vis) S[kb][4 * jj + i] = kNegInf;
          }
    }
    float lsum = 0.f;
#pragma unroll
    for (int g8 = 0; g8 < 8; ++g8) soft_group(g8 >> 2, g8 & 3, lsum);
    if (__builtin_amdgcn_ballot_w64(lsum > kSumLimit || m_run == kNegInf)) {
      float mx = kNegInf;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[kb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = m_new == kNegInf ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_use) * c);
      m_run = m_use;
      nmc = -m_use * c;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) O[db] *= alpha;
      lsum = 0.f;
#pragma unroll
      for (int g8 = 0; g8 < 8; ++g8) soft_group(g8 >> 2, g8 & 3, lsum);
    }
    l_run += lsum;
  };

  // Matrix phase X: Q.K^T of tile t from stage SK into S (if QK_) and P.V of
  // tile t - 1 from stage SV (if PV_), one MFMA of each in turn, operands two
  // ahead.  With ti >= 0 the wave issues its share of ring group ti halfway
  // through the phase.
  auto xphase = [&](auto SK_, auto QK_, auto PV_, int ti) __attribute__((always_inline)) {
    constexpr int SK = decltype(SK_)::value, SV = (SK + kStages - 1) % kStages;
    constexpr bool DO_QK = decltype(QK_)::value, DO_PV = decltype(PV_)::value;
    constexpr int NK = 2 * KS, NV = 4 * DB, NS = NK > NV ? NK : NV;
    constexpr int AH = kOperandsAhead;
    bf16x8 kr[NK], vr[NV];
#pragma unroll
    for (int i = 0; i < AH; ++i) {
      if (DO_QK && i < NK) kr[i] = load_k(i >> 1, i & 1, SK);
      if (DO_PV && i < NV) vr[i] = load_v(i / DB, i % DB, SV);
    }
#if GLANCE_XPRIO
    __builtin_amdgcn_s_setprio(1);
#endif
#pragma unroll
    for (int idx = 0; idx < NS; ++idx) {
      if (DO_QK && idx < NK) {
        if (idx + AH < NK) kr[idx + AH] = load_k((idx + AH) >> 1, (idx + AH) & 1, SK);
        const int ks = idx >> 1, kb = idx & 1;
        S[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kr[idx], qf[ks], ks == 0 ? f32x16{} : S[kb], 0, 0, 0);
      }
      if (DO_PV && idx < NV) {
        if (idx + AH < NV) vr[idx + AH] = load_v((idx + AH) / DB, (idx + AH) % DB, SV);
        const int u = idx / DB, db = idx % DB;
        O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vr[idx], __builtin_bit_cast(bf16x8, Pw[u >> 1][u & 1]),
                                                        O[db], 0, 0, 0);
      }
      if (idx == NS / 2 && ti >= 0) ring_issue(ti);
      __builtin_amdgcn_sched_barrier(0);
    }
#if GLANCE_XPRIO
    __builtin_amdgcn_s_setprio(0);
#endif
  };

  // Schedule.  X_t = {Q.K^T of tile t, P.V of tile t - 1}, Y_t = softmax of
  // tile t; every wave runs barrier 0, X_0 Y_0, barrier 1, X_1 Y_1, ...,
  // X_{n-1} Y_{n-1} and the last P.V.  All waves keep the same order: the two
  // waves of a SIMD drift apart by themselves and overlap one's matrix phase
  // with the other's vector phase, which a fixed rotation of half the waves
  // (lower waves X then Y, upper waves Y then X) did worse, since it put a
  // barrier between the phases of every other wave.
  //
  // Ring invariant: stage s = t % 4 of the ring holds K(t) from its issue
  // right after barrier t - 3 and V(t) from its issue right after barrier
  // t - 2.  K(t) is read in X_t only (between barriers t and t + 1), V(t) in
  // X_{t+1} only (between barriers t + 1 and t + 2).  The issue right after
  // barrier t writes K(t + 3) and V(t + 2) over K(t - 1) and V(t - 2), whose
  // last reads were in X_{t-1}, which every computing wave ended before it
  // arrived at barrier t; and every wave waited for its own share of K(t) and
  // V(t - 1) before it arrived there.  (Waves 4-6 issue group t halfway
  // through X_t rather than right after barrier t: still between barriers t
  // and t + 1, and X_t reads only K(t) and V(t - 1).)
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using YES = std::true_type;
  using NO = std::false_type;
  lds_barrier();  // barrier 0: K(0) has landed, the ancestor words are written
  ring_issue(0);
  xphase(I0{}, YES{}, NO{}, -1);
  auto step = [&](int t, auto SK_) __attribute__((always_inline)) {
    yphase(t - 1);
    ring_wait(t);   // this wave's own share of K(t) and V(t - 1) is complete
    lds_barrier();  // barrier t: every wave's is, and X_{t-1} has ended everywhere
    // group t: waves 0-3 issue right away, waves 4-6 halfway through X_t, so
    // that of the two computing waves sharing a SIMD one computes while the
    // other waits for the memory pipeline to take its loads
    if (wave < 4) ring_issue(t);
    xphase(SK_, YES{}, YES{}, wave < 4 ? -1 : t);
  };
  int t = 1;
  while (t < n_tiles) {
    step(t, I1{});
    if (++t >= n_tiles) break;
    step(t, I2{});
    if (++t >= n_tiles) break;
    step(t, I3{});
    if (++t >= n_tiles) break;
    step(t, I0{});
    ++t;
  }
  yphase(n_tiles - 1);
  switch (n_tiles & 3) {  // P.V of the last tile, stage (n_tiles - 1) % 4
    case 1: xphase(I1{}, NO{}, YES{}, -1); break;
    case 2: xphase(I2{}, NO{}, YES{}, -1); break;
    case 3: xphase(I3{}, NO{}, YES{}, -1); break;
    default: xphase(I0{}, NO{}, YES{}, -1); break;
  }

  l_run += __shfl_xor(l_run, 32);  // lanes l and l + 32 hold the same row
  float M = m_run * c;             // reference in log2 units
  float lsum = l_run;

  if (split) {
    // Partial of this piece in fp16, in the MFMA layout (four values per lane
    // per store, 512 bytes per wave-wide store): the row's O / sum, scaled by
    // 2^-e, 2^e the smallest power of two above its largest |O| / sum, so
    // every stored value lies in (-1, 1) and keeps 11 bits relative to the
    // row's largest, whatever the range of V.  The row's pair becomes
    // (max * c + log2 sum + e, 2^-e): 2^(max * c) sum and O / sum are kept,
    // so the merge's weights and the log-sum-exp are those of the unscaled
    // partial.  O / sum is a convex combination of V rows, so 2^e stays
    // within fp32; e >= -100 keeps 2^-e, and the merge's sum of up to a few
    // hundred of them, finite.  A row with no visible key keeps (-inf, 0).
    float amax = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) amax = fmaxf(amax, fabsf(O[db][i]));
    amax = fmaxf(amax, __shfl_xor(amax, 32));  // lanes l and l + 32 hold the same row
    const float linv = lsum > 0.f ? 1.f / lsum : 0.f;
    const float rmax = amax * linv;
    const int e = rmax > 0.f ? max(__builtin_amdgcn_frexp_expf(rmax), -100) : 0;  // rmax = f 2^e, f in [0.5, 1)
    const float p2 = __builtin_amdgcn_ldexpf(1.f, -e);
    const float sc = linv * p2;
    const size_t ws = ((size_t)g * p.slots_per_g + pc.first + pc.index) * p.row_groups + rgi;
    f16x4* po = reinterpret_cast<f16x4*>(p.part_o) + (ws * p.tiles_rg + wave) * (OV / 4) * 64 + lane;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        po[(db * 4 + j) * 64] = f16x4{(_Float16)(O[db][4 * j] * sc), (_Float16)(O[db][4 * j + 1] * sc),
                                      (_Float16)(O[db][4 * j + 2] * sc), (_Float16)(O[db][4 * j + 3] * sc)};
    if (h == 0)
      p.part_ml[ws * p.rows_rg + 32 * wave + r32] =
          lsum > 0.f ? make_float2(M + __builtin_amdgcn_logf(lsum) + (float)e, p2) : make_float2(M, 0.f);
    return;
  }

  // output: lane l holds O^T[32 db + 8 j + 4 h + i][row], i = 0..3 consecutive dims
  if (!row_ok) return;
  const float inv = 1.f / lsum;
  __bf16* op = static_cast<__bf16*>(p.out) + out_row * D + 4 * h;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bf16x4 o = {(__bf16)(O[db][4 * j] * inv), (__bf16)(O[db][4 * j + 1] * inv),
                        (__bf16)(O[db][4 * j + 2] * inv), (__bf16)(O[db][4 * j + 3] * inv)};
      *reinterpret_cast<bf16x4*>(op + 32 * db + 8 * j) = o;
    }
  if (p.lse && h == 0) p.lse[out_row] = (M + __builtin_amdgcn_logf(lsum)) * kLn2;
}

int grid_blocks(const AttnParams& p) {
  const int slots = p.slots_per_g * p.hkv;
  return ((slots + 7) / 8) * 8 * p.row_groups;
}

}  // namespace

hipError_t launch_attn_bf16(const AttnParams& p, bool tree, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const dim3 grid(grid_blocks(p)), block(512);
  if (ev0) (void)hipEventRecord(ev0, s);
  if (p.d == 128) {
    if (tree) hipLaunchKernelGGL((attn_bf16<128, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_bf16<128, false>), grid, block, 0, s, p);
  } else {
    if (tree) hipLaunchKernelGGL((attn_bf16<64, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((attn_bf16<64, false>), grid, block, 0, s, p);
  }
  hipError_t e = hipGetLastError();
  if (ev1) (void)hipEventRecord(ev1, s);
  return e;
}

}  // namespace glance
