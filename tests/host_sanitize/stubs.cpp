// Host-only stand-ins for the kernel launchers of libglance, for the
// sanitizer build of the host layer (glance_api.cpp).  Each launcher checks
// that every buffer the real kernels would write lies inside the memory the
// host layer handed over (the workspace carve-up against the kernels'
// largest index), records the call and launches nothing.
#include <stdio.h>
#include <stdlib.h>

#include "glance_internal.h"
#include "stubs.h"

StubLog g_stub;

namespace {
// [p, p + bytes) must lie in the recorded workspace.
void in_ws(const void* p, size_t bytes, const char* what) {
  const char* a = static_cast<const char*>(p);
  const char* w = static_cast<const char*>(g_stub.ws);
  if (!w || a < w || a + bytes > w + g_stub.ws_bytes) {
    fprintf(stderr, "STUB FAIL: %s [%p, +%zu) outside the workspace [%p, +%zu)\n", what, p, bytes, (void*)w,
            g_stub.ws_bytes);
    abort();
  }
}
}  // namespace

namespace glance {

hipError_t launch_attn_bf16(const AttnParams& p, bool tree, hipStream_t, hipEvent_t ev0, hipEvent_t ev1) {
  ++g_stub.attn_bf16;
  g_stub.tree = tree;
  g_stub.ev0 = ev0;
  g_stub.ev1 = ev1;
  // the kernels' largest indices: plan[b], part_ml[ws rows_rg + row],
  // part_o[(ws tiles_rg + wave) (D / 8) 64 + lane + ...] fp16 quads (8 bytes)
  const size_t wslots = (size_t)p.slots_per_g * p.hkv * p.row_groups;
  in_ws(p.plan, (size_t)p.batch * sizeof(int2), "piece table");
  in_ws(p.part_ml, wslots * p.rows_rg * sizeof(float2), "(max, sum) partials");
  in_ws(p.part_o, wslots * p.tiles_rg * (size_t)(p.d / 8) * 64 * 8, "output partials");
  if (p.tiles_rg < 1 || p.tiles_rg > 7 || p.rows_rg != 32 * p.tiles_rg) abort();
  if ((long long)p.row_groups * p.rows_rg < p.rows) abort();
  if (p.slots_per_g < p.batch) abort();
  return hipSuccess;
}

hipError_t launch_attn_f32(const AttnParams& p, bool tree, hipStream_t, hipEvent_t ev0, hipEvent_t ev1) {
  ++g_stub.attn_f32;
  g_stub.tree = tree;
  g_stub.ev0 = ev0;
  g_stub.ev1 = ev1;
  const size_t slots = (size_t)p.batch * p.hkv * p.nsplit * p.rows_pad;
  in_ws(p.part_ml, slots * sizeof(float2), "(max, sum) partials");
  in_ws(p.part_o, slots * p.d * sizeof(float), "output partials");
  if ((long long)p.nsplit * p.split_keys < p.cap) abort();
  return hipSuccess;
}

hipError_t launch_attn_merge(const AttnParams&, bool, hipStream_t) {
  ++g_stub.merge;
  return hipSuccess;
}

hipError_t launch_attn_merge_pieces(const AttnParams&, hipStream_t) {
  ++g_stub.merge;
  return hipSuccess;
}

hipError_t launch_accept(const AcceptParams& p, bool, hipStream_t, hipEvent_t ev0, hipEvent_t ev1) {
  ++g_stub.accept;
  g_stub.ev0 = ev0;
  g_stub.ev1 = ev1;
  in_ws(p.part, (size_t)p.batch * p.n_nodes * p.chunks * sizeof(unsigned long long), "chunk words");
  if (p.root_entropy) in_ws(p.ent_part, (size_t)p.batch * p.chunks * sizeof(float4), "entropy chunks");
  if ((long long)p.chunks * p.chunk_len < p.vocab || p.chunk_len % 8) abort();
  return hipSuccess;
}

hipError_t launch_sample(const AcceptParams& p, bool, hipStream_t, hipEvent_t, hipEvent_t) {
  ++g_stub.sample;
  in_ws(p.part, (size_t)p.batch * p.n_nodes * p.chunks * sizeof(unsigned long long), "draw words");
  if ((long long)p.chunks * p.chunk_len < p.vocab) abort();
  return hipSuccess;
}

hipError_t launch_tree(const TreeParams& p, bool, hipStream_t, hipEvent_t, hipEvent_t) {
  ++g_stub.tree_calls;
  if (p.k < 1 || p.k > p.budget || p.slices * kTreeSlice < p.vocab) abort();
  return hipSuccess;
}

hipError_t launch_commit(const CommitParams&, hipStream_t, hipEvent_t, hipEvent_t) {
  ++g_stub.commit;
  return hipSuccess;
}

size_t noalloc_scratch_bytes() { return size_t(1) << 20; }

hipError_t noalloc_scratch(void** out) {
  static unsigned char buf[size_t(1) << 20];
  *out = buf;
  g_stub.ws = buf;
  g_stub.ws_bytes = sizeof(buf);
  return hipSuccess;
}

}  // namespace glance

extern "C" const char* hipGetErrorString(hipError_t) { return "stubbed HIP error"; }
