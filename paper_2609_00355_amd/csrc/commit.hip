// Commit of a round's accepted path into the context cache.  The walk of
// Def. 1 commits the pending root and the accepted tokens (Eq. 1); the verify
// pass computed their keys and values at positions ctx + depth, which for the
// path's nodes are exactly their slots in the prefix.  Cache slot ctx_b + i
// receives the key and value rows of path node i (i = 0..a), then ctx_b grows
// by the rows committed.
//
// One workgroup per sequence: thread 0 resolves the path (clamps, first
// invalid entry) into LDS, every thread copies 16-byte pieces of the rows (or
// single elements when rows are not 16-byte multiples), and the length is
// advanced after a barrier, so no other workgroup ever reads it mid-update.
#include "glance_internal.h"

namespace glance {
namespace {

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr int kCommitThreads = 256;

__global__ __launch_bounds__(kCommitThreads) void commit_kernel(CommitParams p) {
  __shared__ int s_node[64];
  __shared__ int s_rows, s_ctx;
  const int b = blockIdx.x, tid = threadIdx.x;
  if (tid == 0) {
    const int ctx = min(max(p.ctx_lens[b], 0), p.cap);
    const int a = p.accept_len[b];
    int rows = min(min(a + 1, p.path_stride), p.n);
    rows = max(rows, 0);
    int r = 0;
    for (; r < rows; ++r) {
      const int node = p.accept_path[(size_t)b * p.path_stride + r];
      if (node < 0 || node >= p.n) break;
      s_node[r] = node;
    }
    s_rows = r;
    s_ctx = ctx;
  }
  __syncthreads();
  const int rows = s_rows, ctx = s_ctx;
  const int writable = max(0, min(rows, p.cap - ctx));
  const int hkv = p.hkv;
  if (p.vec) {
    const int units = p.d * p.esz / 16;  // 16-byte pieces per (row, head)
    const int per = writable * hkv * units;
    for (int u = tid; u < 2 * per; u += kCommitThreads) {
      const bool is_v = u >= per;
      const int w = is_v ? u - per : u;
      const int piece = w % units, h = (w / units) % hkv, i = w / (units * hkv);
      const size_t src = (((size_t)b * p.n + s_node[i]) * hkv + h) * units + piece;
      const size_t dst = (((size_t)b * hkv + h) * p.cap + ctx + i) * units + piece;
      const u32x4* s = static_cast<const u32x4*>(is_v ? p.v_new : p.k_new);
      u32x4* d = static_cast<u32x4*>(is_v ? p.v_ctx : p.k_ctx);
      d[dst] = s[src];
    }
  } else {
    const int per = writable * hkv * p.d;
    for (int u = tid; u < 2 * per; u += kCommitThreads) {
      const bool is_v = u >= per;
      const int w = is_v ? u - per : u;
      const int e = w % p.d, h = (w / p.d) % hkv, i = w / (p.d * hkv);
      const size_t src = (((size_t)b * p.n + s_node[i]) * hkv + h) * p.d + e;
      const size_t dst = (((size_t)b * hkv + h) * p.cap + ctx + i) * p.d + e;
      if (p.esz == 2) {
        const unsigned short* s = static_cast<const unsigned short*>(is_v ? p.v_new : p.k_new);
        static_cast<unsigned short*>(is_v ? p.v_ctx : p.k_ctx)[dst] = s[src];
      } else {
        const float* s = static_cast<const float*>(is_v ? p.v_new : p.k_new);
        static_cast<float*>(is_v ? p.v_ctx : p.k_ctx)[dst] = s[src];
      }
    }
  }
  __syncthreads();
  if (tid == 0) p.ctx_lens[b] = min(ctx + rows, p.cap);
}

}  // namespace

hipError_t launch_commit(const CommitParams& p, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (ev0) (void)hipEventRecord(ev0, s);
  hipLaunchKernelGGL(commit_kernel, dim3((unsigned)p.batch), dim3(kCommitThreads), 0, s, p);
  const hipError_t e = hipGetLastError();
  if (ev1) (void)hipEventRecord(ev1, s);
  return e;
}

}  // namespace glance
