// Greedy acceptance: the target-greedy token of every verified row and the
// walk of Algorithm 1 (App. B) over the packed tree.
//
// argmax_partial  grid (row, vocabulary chunk): each workgroup streams one
//                 chunk of one row with 16-byte loads and reduces it to a
//                 packed (order key, ~index) word, so that the maximum word
//                 is the largest value at the lowest index.
// accept_walk     one wave per sequence: lane v merges the chunk words of row
//                 v, then the wave walks the tree from the root, finding the
//                 child that carries the current row's argmax token with one
//                 ballot per step.
//
// sample_partial  the sampling walk's row draws (temperature T > 0): the same
//                 grid and packed reduction as argmax_partial over
//                 z / T + g instead of z, with Gumbel noise g = -ln(-ln u);
//                 accept_walk then walks the draws.  u comes from
//                 Philox4x32-10 (Salmon et al., SC'11) with key (seed) and
//                 counter (w / 4, node, sequence, round), word w % 4, mapped
//                 to ((x >> 9) + 0.5) 2^-23; both logarithms use one fixed
//                 fp32 recipe (exponent, then 2 atanh(s) with
//                 s = (m - 1) / (m + 1) as an odd series to s^9) with fused
//                 multiply-add disabled, so every draw is reproducible bit for
//                 bit off the GPU.  Tokens that provably cannot win skip the
//                 logarithms (see sample_partial).
//
// Root entropy (optional): the target's next-token entropy at the round root,
// H = -sum_w p(w) log p(w) over row 0 of each sequence (the scalar of the
// paper's entropy law, Sec. 4).  The argmax workgroups of row 0 re-read their
// chunk (1/n_nodes of the logits) to accumulate, relative to the chunk
// maximum m found by the argmax, S = sum e^(z - m) and T = sum e^(z - m) (z - m);
// the walk merges the chunks to H = log S - T / S.
//
// Order key of a float (fp32 bits, or bf16 bits shifted up 16): the sign-
// magnitude encoding mapped to two's complement, so +0 and -0 both map to 0
// (they tie, and the lowest index wins), and every NaN maps to INT32_MAX (a
// NaN is larger than every number; the first NaN wins).
#include "glance_internal.h"

namespace glance {
namespace {

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

__device__ __forceinline__ int order_key(unsigned int bits) {
  const int neg = (int)(0x80000000u - bits);  // -(magnitude) for a negative value
  int k = ((int)bits < 0) ? neg : (int)bits;
  // a NaN: magnitude above +inf; positive NaN already exceeds +inf, negative NaN does not
  k = ((bits & 0x7fffffffu) > 0x7f800000u) ? 0x7fffffff : k;
  return k;
}

__device__ __forceinline__ unsigned long long pack(int key, int idx) {
  return ((unsigned long long)((unsigned int)key ^ 0x80000000u) << 32) |
         (unsigned long long)(0xffffffffu - (unsigned int)idx);
}

// Inverse of order_key for a non-NaN key: the fp32 bits of the value.
__device__ __forceinline__ float key_to_float(int key) {
  const unsigned bits = key >= 0 ? (unsigned)key : 0x80000000u - (unsigned)key;
  return __builtin_bit_cast(float, bits);
}

__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) {
  return a > b ? a : b;
}

__device__ __forceinline__ unsigned long long wave_max64(unsigned long long v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const unsigned int lo = __shfl_xor((unsigned int)v, off);
    const unsigned int hi = __shfl_xor((unsigned int)(v >> 32), off);
    v = umax64(v, ((unsigned long long)hi << 32) | lo);
  }
  return v;
}

__device__ __forceinline__ float as_f32(unsigned u) { return __builtin_bit_cast(float, u); }

// IEEE 754-2019 maximum (v_maximum3_f32): a NaN operand gives NaN, and -0 < +0.
__device__ __forceinline__ float fmaximum(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float fmaximum3(float a, float b, float c) { return fmaximum(fmaximum(a, b), c); }

// bf16 rows with 16-byte alignment.  A 32-bit word w holds two bf16 values:
// the high one read as fp32 is w itself (the low value only adds mantissa
// bits below the bf16 precision, so the order of distinct bf16 values is
// kept), the low one is w << 16.  Per 8 values the thread takes one fp32
// maximum, masks it back to bf16 precision and keeps the first 8-value vector
// that reached its running best, together with that vector itself, so the
// lowest index holding the best value is found at the end without a second
// read.  The maximum propagates NaN, so a chunk holding a NaN (or an infinity,
// which the extra mantissa bits can turn into a NaN) shows up as a NaN running
// maximum; such chunks, and chunks whose best value is +0 or -0 (which must
// tie), are redone by the exact scalar scan.
__device__ __forceinline__ void argmax_bf16_fast(const unsigned short* x, int c0, int c1, int tid,
                                                 int& best_key, int& best_idx) {
  constexpr int kUnroll = 8;
  constexpr unsigned kPad = 0xff7fff7fu;  // two finite -3.39e38 values, never selected
  float bk = -__builtin_inff();
  float run = -__builtin_inff();
  int bpos = -1;
  u32x4 bv = {0u, 0u, 0u, 0u};
  for (int e0 = c0 + 8 * tid; e0 < c1; e0 += 8 * 256 * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int e = e0 + u * 8 * 256;
      v[u] = e < c1 ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(x + e))
                    : u32x4{kPad, kPad, kPad, kPad};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int e = e0 + u * 8 * 256;
      const float a = fmaximum3(as_f32(v[u][0]), as_f32(v[u][1]), as_f32(v[u][2]));
      const float b = fmaximum3(as_f32(v[u][3]), as_f32(v[u][0] << 16), as_f32(v[u][1] << 16));
      const float m = fmaximum3(as_f32(v[u][2] << 16), as_f32(v[u][3] << 16), fmaximum(a, b));
      run = fmaximum(run, m);
      const float vm = as_f32(__builtin_bit_cast(unsigned, m) & 0xffff0000u);
      if ((vm > bk || bpos < 0) && e < c1) { bk = vm; bpos = e; bv = v[u]; }
    }
  }
  const bool redo = run != run || bk == 0.f;
  if (__syncthreads_or(redo)) {  // exact path: NaN is the largest value, the first one wins
    for (int e = c0 + tid; e < c1; e += 256) {
      const int k = order_key((unsigned int)x[e] << 16);
      if (k > best_key) { best_key = k; best_idx = e; }
    }
    return;
  }
  if (bpos < 0) return;
  unsigned bits = 0;
#pragma unroll
  for (int w = 3; w >= 0; --w) {  // backwards, so the lowest index overwrites last
    if (as_f32(bv[w] & 0xffff0000u) == bk) { best_idx = bpos + 2 * w + 1; bits = bv[w] >> 16; }
    if (as_f32(bv[w] << 16) == bk) { best_idx = bpos + 2 * w; bits = bv[w] & 0xffffu; }
  }
  best_key = order_key(bits << 16);
}

template <bool BF16, bool VEC>
__global__ __launch_bounds__(256) void argmax_partial(AcceptParams p) {
  __shared__ unsigned long long red[4];
  const int chunk = blockIdx.x % p.chunks;
  const long row = blockIdx.x / p.chunks;
  const int c0 = chunk * p.chunk_len;
  const int c1 = min(p.vocab, c0 + p.chunk_len);
  const int tid = threadIdx.x;
  int best_key = (int)0x80000000;
  int best_idx = 0x7fffffff;
  if (BF16) {
    const unsigned short* x = static_cast<const unsigned short*>(p.logits) + row * (long)p.vocab;
    if (VEC) {
      argmax_bf16_fast(x, c0, c1, tid, best_key, best_idx);
    } else {
      for (int e = c0 + tid; e < c1; e += 256) {
        const int k = order_key((unsigned int)x[e] << 16);
        if (k > best_key) { best_key = k; best_idx = e; }
      }
    }
  } else {
    const unsigned int* x = static_cast<const unsigned int*>(p.logits) + row * (long)p.vocab;
    if (VEC) {
      constexpr int kUnroll = 4;
      for (int e0 = c0 + 4 * tid; e0 < c1; e0 += 4 * 256 * kUnroll) {
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int e = e0 + u * 4 * 256;
          v[u] = e < c1 ? *reinterpret_cast<const u32x4*>(x + e) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int e = e0 + u * 4 * 256;
          if (e >= c1) break;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int k = order_key(v[u][w]);
            if (k > best_key) { best_key = k; best_idx = e + w; }
          }
        }
      }
    } else {
      for (int e = c0 + tid; e < c1; e += 256) {
        const int k = order_key(x[e]);
        if (k > best_key) { best_key = k; best_idx = e; }
      }
    }
  }
  // threads that saw no element keep the smallest possible word
  unsigned long long w = (best_idx == 0x7fffffff) ? 0ull : pack(best_key, best_idx);
  w = wave_max64(w);
  if ((tid & 63) == 0) red[tid >> 6] = w;
  __syncthreads();
  __shared__ float ent[2][4];
  __shared__ float s_m;
  if (tid == 0) {
    const unsigned long long r = umax64(umax64(red[0], red[1]), umax64(red[2], red[3]));
    p.part[row * p.chunks + chunk] = r;
    s_m = key_to_float((int)((unsigned)(r >> 32) ^ 0x80000000u));
  }
  if (p.root_entropy == nullptr || row % p.n_nodes != 0) return;
  // root row: entropy statistics of the chunk relative to its maximum
  __syncthreads();
  const float m = s_m;
  float S = 0.f, T = 0.f;
  for (int e = c0 + tid; e < c1; e += 256) {
    const float z = BF16 ? __builtin_bit_cast(float, (unsigned)static_cast<const unsigned short*>(p.logits)[row * (long)p.vocab + e] << 16)
                         : static_cast<const float*>(p.logits)[row * (long)p.vocab + e];
    if (z != -__builtin_inff()) {
      const float d = z - m;
      const float x = __builtin_amdgcn_exp2f(d * 1.4426950408889634f);
      S += x;
      T += x * d;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    S += __shfl_xor(S, off);
    T += __shfl_xor(T, off);
  }
  if ((tid & 63) == 0) {
    ent[0][tid >> 6] = S;
    ent[1][tid >> 6] = T;
  }
  __syncthreads();
  if (tid == 0) {
    const float s_all = (ent[0][0] + ent[0][1]) + (ent[0][2] + ent[0][3]);
    const float t_all = (ent[1][0] + ent[1][1]) + (ent[1][2] + ent[1][3]);
    p.ent_part[(row / p.n_nodes) * p.chunks + chunk] = make_float4(m, s_all, t_all, 0.f);
  }
}

// Philox4x32-10: ten rounds of two 32x32 -> 64-bit multiplies and a
// counter shuffle, the key advanced by the Weyl constants between rounds.
__device__ __forceinline__ void philox4x32_10(unsigned (&c)[4], unsigned k0, unsigned k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const unsigned long long p0 = (unsigned long long)0xD2511F53u * c[0];
    const unsigned long long p1 = (unsigned long long)0xCD9E8D57u * c[2];
    // three-input XOR in one v_bitop3_b32 (truth table 0x96)
    const unsigned n0 = __builtin_amdgcn_bitop3_b32((unsigned)(p1 >> 32), c[1], k0, 0x96);
    const unsigned n2 = __builtin_amdgcn_bitop3_b32((unsigned)(p0 >> 32), c[3], k1, 0x96);
    c[0] = n0;
    c[1] = (unsigned)p1;
    c[2] = n2;
    c[3] = (unsigned)p0;
  }
}

// ln t for a positive normal t by the fixed recipe: t = m 2^e with m in
// [sqrt(1/2), sqrt(2)) (so m - 1 is exact and t near 1 keeps e = 0), then
// e ln 2 + 2 atanh(s), s = (m - 1) / (m + 1), atanh(s) / s as the series
// 1 + s^2/3 + ... + s^8/9.  IEEE-rounded operations, no fused multiply-add.
__device__ __forceinline__ float ln_fixed(float t) {
#pragma clang fp contract(off)
  const unsigned bits = __builtin_bit_cast(unsigned, t);
  const unsigned mant = bits & 0x007FFFFFu;
  const bool high = mant > 0x3504F3u;  // m >= sqrt(2): halve it
  const int e = (int)((bits >> 23) & 0xFFu) - 127 + (high ? 1 : 0);
  const float m = __builtin_bit_cast(float, mant | (high ? 0x3F000000u : 0x3F800000u));
  const float s = (m - 1.0f) / (m + 1.0f);
  const float s2 = s * s;
  float acc = (float)(1.0 / 9.0);
  acc = acc * s2 + (float)(1.0 / 7.0);
  acc = acc * s2 + (float)(1.0 / 5.0);
  acc = acc * s2 + (float)(1.0 / 3.0);
  acc = acc * s2 + 1.0f;
  const float at2 = 2.0f * (s * acc);
  return (float)e * (float)0.6931471805599453 + at2;
}

// The perturbed logit z / T + g of one token, g = -ln(-ln u), exactly as the
// definition rounds it.
__device__ __forceinline__ float gumbel_logit(float z, float temperature, unsigned x) {
#pragma clang fp contract(off)
  const float u = ((float)(x >> 9) + 0.5f) * 0x1p-23f;
  const float g = -ln_fixed(-ln_fixed(u));
  return z / temperature + g;
}

// Monotone map between floats and signed integers (its own inverse): larger
// numbers give larger keys; a positive NaN maps above +inf.
__device__ __forceinline__ int float_order(int bits) { return bits ^ ((bits >> 31) & 0x7fffffff); }

// Wave maximum of integer keys, broadcast; every lane must be active.
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp_i(int v) {  // lanes a row mask leaves out read INT_MIN
  return __builtin_amdgcn_update_dpp((int)0x80000000, v, CTRL, ROWS, 0xf, false);
}
__device__ __forceinline__ int wave_max_key(int v) {
  v = max(v, dpp_i<0xb1, 0xf>(v));
  v = max(v, dpp_i<0x4e, 0xf>(v));
  v = max(v, dpp_i<0x141, 0xf>(v));
  v = max(v, dpp_i<0x140, 0xf>(v));
  v = max(v, dpp_i<0x142, 0xa>(v));
  v = max(v, dpp_i<0x143, 0xc>(v));
  return __builtin_amdgcn_readlane(v, 63);
}

// One group of four tokens as raw words (bf16 pairs, or fp32 bits), loaded a
// loop iteration ahead and unpacked when used.
template <bool BF16, bool VEC>
__device__ __forceinline__ void load_group(const void* rowp, int e4, unsigned (&w)[4]) {
  if (BF16) {
    const unsigned short* x = static_cast<const unsigned short*>(rowp);
    if (VEC) {
      const uint2 v = *reinterpret_cast<const uint2*>(x + e4);
      w[0] = v.x;
      w[1] = v.y;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = x[e4 + j];
    }
  } else {
    const unsigned* x = static_cast<const unsigned*>(rowp);
    if (VEC) {
      const uint4 v = *reinterpret_cast<const uint4*>(x + e4);
      w[0] = v.x;
      w[1] = v.y;
      w[2] = v.z;
      w[3] = v.w;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = x[e4 + j];
    }
  }
}

template <bool BF16, bool VEC>
__device__ __forceinline__ void unpack_group(const unsigned (&w)[4], float (&z)[4]) {
  if (BF16 && VEC) {
    z[0] = __builtin_bit_cast(float, w[0] << 16);
    z[1] = __builtin_bit_cast(float, w[0] & 0xffff0000u);
    z[2] = __builtin_bit_cast(float, w[1] << 16);
    z[3] = __builtin_bit_cast(float, w[1] & 0xffff0000u);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) z[j] = __builtin_bit_cast(float, BF16 ? w[j] << 16 : w[j]);
  }
}

// Row draws of the sampling walk.  Evaluating both logarithms for every token
// would cost about a hundred instructions a token, so each token is first
// tested against the wave's running best y* (the largest z / T + g found so
// far by any lane of the wave) with an upper bound on its noise read off the
// uniform's integer: with u = (k + 0.5) 2^-23, r = 2^23 - 1 - k and x the
// generator word (k = x >> 9), g <= -ln(1 - u) <= (23 - log2 r) ln 2, and
// log2 r >= F 2^-23 - 127 with F the fp32 bits of float(r) (its exponent plus
// mantissa fraction, since log2(1 + f) >= f on [0, 1]); on average the bound
// sits within 0.46 of the noise, and the fixed recipe stays below it.  A token is skipped only when
// z / T plus that bound plus a margin for every rounding involved (2^-17
// relative, 2^-12 absolute) is still below y*: then a strictly larger value
// exists and the token cannot be the draw.  Before the generator runs, the
// largest bound, 24 ln 2, tests the group's largest logit (NaN-propagating)
// to skip whole groups of four.  -inf logits are clamped to -FLT_MAX for the
// group test, so fully masked groups are skipped once y* is finite.  Survivors take the
// exact definition.  (A -inf logit inside a group with finite ones gives a NaN
// bound and takes the exact path: slower, never wrong.)
struct SampleState {
  int best_key, best_idx;
  float lane_best;  // y of the lane's best token
};

// One group of four tokens of one lane.  FIRST (the wave's first full
// group, no running best yet): the wave first takes the largest lower bound
// on z / T + g over its 256 tokens as y*, from the integer alone: for
// u >= 1/2, -ln u <= (1 - u) / u gives g >= -ln(1 - u) - 2 (1 - u), bounded
// below through the fp32 bits of float(r + 1) (within about 0.05 of the
// noise in its upper tail); g >= -2.82 for u < 1/2; less the same rounding
// allowance.  Every value is at most some token's exact z / T + g, and the
// token reaching it is never skipped, so the exact draw is kept.
template <bool TAIL, bool FIRST>
__device__ __forceinline__ void sample_group(const AcceptParams& p, const float (&z)[4], int e4, int c1,
                                             unsigned node, unsigned seq, unsigned rnd, float& wbest,
                                             SampleState& st) {
  constexpr float kLn2 = 0.6931472f;
  const float inv_t = p.inv_temperature;
  if (!FIRST) {
    // group test with the largest bound
    const float slack = fmaf(fabsf(wbest), 0x1p-17f, 0x1p-12f);
    float m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(z[0], z[1]),
                                            __builtin_elementwise_maximum(z[2], z[3]));
    float mt = m * inv_t;
    mt = mt == -__builtin_inff() ? -3.4028234663852886e38f : mt;
    const bool group_beaten = fmaf(fabsf(mt), 0x1p-17f, mt) + (slack + 24.f * kLn2) < wbest;
    if (group_beaten && !TAIL) return;
    if (TAIL && (group_beaten || e4 >= c1)) return;
  }
  unsigned c[4] = {(unsigned)e4 >> 2, node, seq, rnd};
  philox4x32_10(c, p.seed_lo, p.seed_hi);
  if (FIRST) {
    int lo_key = (int)0x80000000;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float zt = z[j] * inv_t;
      const float zt_lo = zt * (zt >= 0.f ? 1.0f - 0x1p-17f : 1.0f + 0x1p-17f);
      // r + 1 = 2^23 - k; log2(r + 1) <= F 2^-23 - 127 + 0.0861 for F the bits of float(r + 1)
      const float r1 = (float)(0x800000u - (c[j] >> 9));
      const float lg1 = (float)__builtin_bit_cast(unsigned, r1) * 0x1p-23f - 127.f;
      const float g_lo = (int)c[j] < 0 ? (22.9138f - lg1) * kLn2 - 2.f * (r1 * 0x1p-23f) : -2.82f;
      lo_key = max(lo_key, float_order(__builtin_bit_cast(int, zt_lo + g_lo - 0x1p-12f)));
    }
    wbest = __builtin_bit_cast(float, float_order(wave_max_key(lo_key)));
  }
  const float slack = fmaf(fabsf(wbest), 0x1p-17f, 0x1p-12f);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (TAIL && e4 + j >= c1) break;
    const float zt = z[j] * inv_t;
    // upper bound on the noise: g <= -ln(1 - u) <= (23 - log2 r) ln 2 with
    // r = 2^23 - 1 - k, log2 r bounded below by the fp32 bits of float(r)
    // read as exponent plus mantissa fraction (r = 0: 150 ln 2)
    const unsigned r = 0x7FFFFFu - (c[j] >> 9);
    const float lg2r = (float)__builtin_bit_cast(unsigned, (float)r) * 0x1p-23f - 127.f;
    const float bound = fmaf(23.f - lg2r, kLn2, fmaf(fabsf(zt), 0x1p-17f, zt) + slack);
    if (!(bound < wbest)) {
      const float y = gumbel_logit(z[j], p.temperature, c[j]);
      const int k = order_key(__builtin_bit_cast(unsigned, y));
      if (k > st.best_key) {
        st.best_key = k;
        st.best_idx = e4 + j;
        st.lane_best = y;
      }
    }
  }
}

template <bool BF16, bool VEC>
__global__ __launch_bounds__(256) void sample_partial(AcceptParams p) {
  __shared__ unsigned long long red[4];
  __shared__ __align__(16) float s_best[4];  // each wave's running best, shared without barriers
  const int chunk = blockIdx.x % p.chunks;
  const long row = blockIdx.x / p.chunks;
  const unsigned node = (unsigned)(row % p.n_nodes), seq = (unsigned)(row / p.n_nodes);
  const int c0 = chunk * p.chunk_len;  // a multiple of 8: groups of four never straddle chunks
  const int c1 = min(p.vocab, c0 + p.chunk_len);
  const int full_end = c0 + (c1 - c0) / 1024 * 1024;  // iterations where every lane has four tokens
  const int tid = threadIdx.x, wave = tid >> 6;
  const char* rowp = static_cast<const char*>(p.logits) + row * (long)p.vocab * (BF16 ? 2 : 4);
  // the round number: the argument, plus the device counter when one is given
  // (the walk kernel, later on the stream, advances it)
  const unsigned rnd = p.round + (p.round_counter ? __hip_atomic_load(p.round_counter, __ATOMIC_RELAXED,
                                                                      __HIP_MEMORY_SCOPE_AGENT)
                                                  : 0u);
  SampleState st = {(int)0x80000000, 0x7fffffff, -__builtin_inff()};
  float wbest = -__builtin_inff();  // a value some token of the workgroup reaches
  if ((tid & 63) == 0) s_best[wave] = -__builtin_inff();
  __syncthreads();
  // A wave publishes its running best to its slot and takes the maximum of
  // the four slots.  Reads may see another wave's older value: every value a
  // slot ever holds is reached by some token, so a stale one only skips less.
  auto share = [&]() __attribute__((always_inline)) {
    const float wm = __builtin_bit_cast(float, float_order(wave_max_key(float_order(__builtin_bit_cast(int, st.lane_best)))));
    wbest = wm > wbest ? wm : wbest;  // a NaN maximum leaves wbest as it is
    if ((tid & 63) == 0) __hip_atomic_store(&s_best[wave], wbest, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    float o = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float x = __hip_atomic_load(&s_best[w], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      o = x > o ? x : o;
    }
    o = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, o)));
    wbest = o > wbest ? o : wbest;
  };
  unsigned wn[4] = {0u, 0u, 0u, 0u};
  if (c0 < full_end) {
    load_group<BF16, VEC>(rowp, c0 + 4 * tid, wn);
    float z[4];
    unpack_group<BF16, VEC>(wn, z);
    if (c0 + 1024 < full_end) load_group<BF16, VEC>(rowp, c0 + 1024 + 4 * tid, wn);
    sample_group<false, true>(p, z, c0 + 4 * tid, c1, node, seq, rnd, wbest, st);
    share();
  }
  // the running best is exchanged every iteration while it still climbs fast,
  // then every fourth (a uniform condition: the exchange needs every lane)
  int it = 0;
  for (int base = c0 + 1024; base < full_end; base += 1024) {  // the same trip count for every lane
    float z[4];
    unpack_group<BF16, VEC>(wn, z);
    if (base + 1024 < full_end) load_group<BF16, VEC>(rowp, base + 1024 + 4 * tid, wn);
    sample_group<false, false>(p, z, base + 4 * tid, c1, node, seq, rnd, wbest, st);
    ++it;
    if (it <= 4 || (it & 3) == 0) share();
  }
  if (full_end < c1) {  // the ragged tail: per-token bounds checks
    const int e4 = full_end + 4 * tid;
    float z[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      z[j] = e4 + j < c1 ? (BF16 ? __builtin_bit_cast(float, (unsigned)reinterpret_cast<const unsigned short*>(rowp)[e4 + j] << 16)
                                 : reinterpret_cast<const float*>(rowp)[e4 + j])
                         : -__builtin_inff();
    sample_group<true, false>(p, z, e4, c1, node, seq, rnd, wbest, st);
  }
  unsigned long long w = (st.best_idx == 0x7fffffff) ? 0ull : pack(st.best_key, st.best_idx);
  w = wave_max64(w);
  if ((tid & 63) == 0) red[tid >> 6] = w;
  __syncthreads();
  if (tid == 0) p.part[row * p.chunks + chunk] = umax64(umax64(red[0], red[1]), umax64(red[2], red[3]));
}

__global__ __launch_bounds__(64) void accept_walk(AcceptParams p) {
  __shared__ int sAm[64];
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int n = p.n_nodes;
  const long rb = (long)b * n;

  int am = 0;
  int par = -1;
  int tok = 0;
  if (lane < n) {
    // the tree and the chunk words are all loaded before any is used (one
    // memory round trip; the argmax store below could alias the tree inputs,
    // so the compiler would not hoist their loads over it)
    par = p.parents[rb + lane];
    tok = p.tokens[rb + lane];
    unsigned long long w = 0ull;
    const unsigned long long* src = p.part + (rb + lane) * p.chunks;
    for (int c0 = 0; c0 < p.chunks; c0 += 8) {
      unsigned long long v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = c0 + u < p.chunks ? src[c0 + u] : 0ull;
#pragma unroll
      for (int u = 0; u < 8; ++u) w = umax64(w, v[u]);
    }
    am = (int)(0xffffffffu - (unsigned int)(w & 0xffffffffull));
    p.argmax_out[rb + lane] = am;
    sAm[lane] = am;
  }
  __syncthreads();

  // Walk: from node v, descend to the lowest-index child c > v of v whose token
  // is argmax(row v).  Node indices strictly increase, so at most n - 1 steps.
  int v = 0;
  int len = 0;
  int32_t* path = p.accept_path + (long)b * p.path_stride;
  if (lane == 0) path[0] = 0;
  for (int step = 0; step < n; ++step) {
    const int t = sAm[v];
    const bool hit = (lane < n) && (lane > v) && (par == v) && (tok == t);
    const unsigned long long m = __ballot(hit);
    if (m == 0ull) break;
    v = __ffsll((long long)m) - 1;
    ++len;
    if (lane == 0 && len < p.path_stride) path[len] = v;
  }
  for (int k = len + 1 + lane; k < p.path_stride; k += 64) path[k] = -1;
  if (lane == 0) {
    p.accept_len[b] = len;
    p.next_root[b] = sAm[v];
  }
  // sampling with a device round counter: every row draw of this call has
  // read it (the draws kernel ran earlier on the stream), so advance it once
  if (p.round_counter && b == 0 && lane == 0) {
    const unsigned r = __hip_atomic_load(p.round_counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p.round_counter, r + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (p.root_entropy && lane == 0) {
    // merge the chunks relative to the row maximum M:
    // e^(z-M) (z-M) = e^(m-M) e^(z-m) ((z-m) + (m-M))
    const float4* ep = p.ent_part + (long)b * p.chunks;
    float M = -__builtin_inff();
    for (int c = 0; c < p.chunks; ++c) M = fmaxf(M, ep[c].x);
    float S = 0.f, T = 0.f;
    for (int c = 0; c < p.chunks; ++c) {
      const float4 q = ep[c];
      if (q.y == 0.f) continue;  // a chunk of -inf logits holds no mass
      const float f = __builtin_amdgcn_exp2f((q.x - M) * 1.4426950408889634f);
      S += q.y * f;
      T += (q.z + (q.x - M) * q.y) * f;
    }
    p.root_entropy[b] = __builtin_amdgcn_logf(S) * 0.6931471805599453f - T / S;
  }
}

}  // namespace

hipError_t launch_sample(const AcceptParams& p, bool bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const long rows = (long)p.batch * p.n_nodes;
  const dim3 grid((unsigned)(rows * p.chunks)), block(256);
  const size_t vbytes = bf16 ? 8 : 16;  // one group of four tokens
  const bool vec = ((size_t)p.vocab * (bf16 ? 2 : 4)) % vbytes == 0 &&
                   (reinterpret_cast<uintptr_t>(p.logits) % vbytes) == 0;
  if (ev0) (void)hipEventRecord(ev0, s);
  if (bf16) {
    if (vec) hipLaunchKernelGGL((sample_partial<true, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((sample_partial<true, false>), grid, block, 0, s, p);
  } else {
    if (vec) hipLaunchKernelGGL((sample_partial<false, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((sample_partial<false, false>), grid, block, 0, s, p);
  }
  hipError_t e = hipGetLastError();
  if (ev1) (void)hipEventRecord(ev1, s);
  if (e != hipSuccess) return e;
  AcceptParams pw = p;
  pw.root_entropy = nullptr;
  hipLaunchKernelGGL(accept_walk, dim3(p.batch), dim3(64), 0, s, pw);
  return hipGetLastError();
}

hipError_t launch_accept(const AcceptParams& p, bool bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const long rows = (long)p.batch * p.n_nodes;
  const dim3 grid((unsigned)(rows * p.chunks)), block(256);
  const size_t esz = bf16 ? 2 : 4;
  const bool vec = ((size_t)p.vocab * esz) % 16 == 0 &&
                   (reinterpret_cast<uintptr_t>(p.logits) & 15) == 0;
  if (ev0) (void)hipEventRecord(ev0, s);
  if (bf16) {
    if (vec) hipLaunchKernelGGL((argmax_partial<true, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((argmax_partial<true, false>), grid, block, 0, s, p);
  } else {
    if (vec) hipLaunchKernelGGL((argmax_partial<false, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((argmax_partial<false, false>), grid, block, 0, s, p);
  }
  hipError_t e = hipGetLastError();
  if (ev1) (void)hipEventRecord(ev1, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_walk, dim3(p.batch), dim3(64), 0, s, p);
  return hipGetLastError();
}

}  // namespace glance
