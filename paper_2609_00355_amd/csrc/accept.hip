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

typedef short s16x2 __attribute__((ext_vector_type(2)));

// Order keys of the two bf16 values packed in w, as int16 lanes, with packed
// 16-bit instructions: sign-magnitude -> two's complement, so +0 and -0 both
// give 0 and every non-NaN value keeps its order.  A NaN gives a key above
// +inf (0x7f80) or below -inf (-0x7f80); such chunks take the exact scalar path.
__device__ __forceinline__ s16x2 key2(unsigned w) {
  const s16x2 x = __builtin_bit_cast(s16x2, w);
  const s16x2 t = x >> (s16x2){15, 15};                       // -1 for negatives, else 0
  const s16x2 k = x ^ (t & (s16x2){0x7fff, 0x7fff});          // negatives -> -1 - magnitude
  return k - t;                                               // negatives -> -magnitude
}

// bf16 rows with 16-byte alignment: per 8 values, the packed keys are reduced
// to one maximum, compared once with the thread's running best, and only the
// position of the 8-value vector that first reached the best is kept.  At the
// end the thread re-reads that one vector to find the lowest index holding
// the best key.  Chunks containing a NaN are redone by the exact scalar scan.
__device__ __forceinline__ void argmax_bf16_fast(const unsigned short* x, int c0, int c1, int tid,
                                                 int& best_key, int& best_idx) {
  constexpr int kUnroll = 4;
  int bk = -0x8000 - 1;  // below every int16 key
  int bpos = -1;
  s16x2 lo = (s16x2){0x7fff, 0x7fff};
  s16x2 hi = (s16x2){-0x7fff, -0x7fff};
  for (int e0 = c0 + 8 * tid; e0 < c1; e0 += 8 * 256 * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int e = e0 + u * 8 * 256;
      v[u] = e < c1 ? *reinterpret_cast<const u32x4*>(x + e) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int e = e0 + u * 8 * 256;
      if (e >= c1) break;
      const s16x2 k0 = key2(v[u][0]), k1 = key2(v[u][1]), k2 = key2(v[u][2]), k3 = key2(v[u][3]);
      const s16x2 mx = __builtin_elementwise_max(__builtin_elementwise_max(k0, k1), __builtin_elementwise_max(k2, k3));
      const s16x2 mn = __builtin_elementwise_min(__builtin_elementwise_min(k0, k1), __builtin_elementwise_min(k2, k3));
      hi = __builtin_elementwise_max(hi, mx);
      lo = __builtin_elementwise_min(lo, mn);
      const int vm = max((int)mx[0], (int)mx[1]);
      if (vm > bk) { bk = vm; bpos = e; }
    }
  }
  const bool nan_seen = max((int)hi[0], (int)hi[1]) > 0x7f80 || min((int)lo[0], (int)lo[1]) < -0x7f80;
  if (__syncthreads_or(nan_seen)) {  // exact path: NaN is the largest value, the first one wins
    for (int e = c0 + tid; e < c1; e += 256) {
      const int k = order_key((unsigned int)x[e] << 16);
      if (k > best_key) { best_key = k; best_idx = e; }
    }
    return;
  }
  if (bpos >= 0) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(x + bpos);
#pragma unroll
    for (int w = 3; w >= 0; --w) {  // backwards, so the lowest index overwrites last
      const s16x2 k = key2(v[w]);
      if (k[1] == bk) best_idx = bpos + 2 * w + 1;
      if (k[0] == bk) best_idx = bpos + 2 * w;
    }
    best_key = order_key((unsigned int)x[best_idx] << 16);
  }
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
  if (tid == 0) {
    const unsigned long long r = umax64(umax64(red[0], red[1]), umax64(red[2], red[3]));
    p.part[row * p.chunks + chunk] = r;
  }
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
    unsigned long long w = 0ull;
    const unsigned long long* src = p.part + (rb + lane) * p.chunks;
    for (int c = 0; c < p.chunks; ++c) w = umax64(w, src[c]);
    am = (int)(0xffffffffu - (unsigned int)(w & 0xffffffffull));
    p.argmax_out[rb + lane] = am;
    par = p.parents[rb + lane];
    tok = p.tokens[rb + lane];
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
}

}  // namespace

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
