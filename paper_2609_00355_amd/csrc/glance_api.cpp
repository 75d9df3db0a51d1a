// C-ABI host layer: argument checks, split-KV planning, workspace layout and
// kernel launches for the GLANCE round hot path (see include/glance.h).
#include "glance.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <string>

#include <cfloat>

#include "glance_internal.h"

namespace {

thread_local std::string g_last_error;
thread_local hipEvent_t g_ev_start = nullptr;
thread_local hipEvent_t g_ev_stop = nullptr;

glance_status fail(glance_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
glance_status fail(glance_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

glance_status ok() { return GLANCE_OK; }

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// fp32 kernel: context keys per split, about one workgroup per compute unit
// over the whole grid, at least 256 and at most 8192 keys per split.
// Context keys per split of the fp32 kernel: about 256 workgroups over the
// capacity, at least one key tile (a workgroup walks its tiles one after
// another, so small shapes finish sooner in more, shorter splits).
int f32_split_keys(const glance_attn_shape& s, int row_groups) {
  const long long cap = s.ctx_capacity > 0 ? s.ctx_capacity : 1;
  long long per = cap * s.batch * s.n_kv_heads * row_groups / 256;
  per = (per + glance::kKeyTile - 1) / glance::kKeyTile * glance::kKeyTile;
  if (per < glance::kKeyTile) per = glance::kKeyTile;
  if (per > 8192) per = 8192;
  return (int)per;
}

// Attention workspace: [piece table][(max, sum) partials][O partials].
struct Plan {
  glance::AttnParams p;
  size_t counter_bytes;  // the bf16 path's per-sequence piece table
  size_t part_ml_bytes;
  size_t part_o_bytes;
  size_t total;
};

// A glance_dtype as the integer the caller stored: a C caller may store any
// int in the field, and reading an out-of-range value as the C++ enum type
// would be undefined, so the bits are copied out and compared as an int.
int dtype_bits(const glance_dtype& d) {
  int v;
  memcpy(&v, &d, sizeof v);
  return v;
}

bool dtype_ok(const glance_dtype& d) {
  const int v = dtype_bits(d);
  return v == GLANCE_F32 || v == GLANCE_BF16;
}

glance_status check_shape(const glance_attn_shape* s) {
  if (!s) return fail(GLANCE_ERR_INVALID_ARG, "shape is NULL");
  if (s->batch < 1) return fail(GLANCE_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", s->batch);
  if (s->n_new < 1 || s->n_new > 64)
    return fail(GLANCE_ERR_UNSUPPORTED, "n_new must be in 1..64 (got %d)", s->n_new);
  if (s->n_kv_heads < 1) return fail(GLANCE_ERR_INVALID_ARG, "n_kv_heads must be >= 1");
  if (s->n_q_heads < 1 || s->n_q_heads % s->n_kv_heads != 0)
    return fail(GLANCE_ERR_INVALID_ARG, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)",
                s->n_q_heads, s->n_kv_heads);
  if (s->n_q_heads / s->n_kv_heads > 16)
    return fail(GLANCE_ERR_UNSUPPORTED, "at most 16 query heads per KV head (got %d)",
                s->n_q_heads / s->n_kv_heads);
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(GLANCE_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", s->head_dim);
  if (s->ctx_capacity < 0) return fail(GLANCE_ERR_INVALID_ARG, "ctx_capacity must be >= 0");
  if (!dtype_ok(s->dtype)) return fail(GLANCE_ERR_UNSUPPORTED, "dtype must be GLANCE_F32 or GLANCE_BF16");
  if (!(s->sm_scale == s->sm_scale) || isinf(s->sm_scale))
    return fail(GLANCE_ERR_INVALID_ARG, "sm_scale must be finite");
  // index arithmetic in the kernels: element offsets fit in 64 bits, per-tensor
  // row counts in 32 bits
  const long long rows = (long long)s->batch * s->n_new * s->n_q_heads;
  if (rows > 0x3fffffffLL) return fail(GLANCE_ERR_UNSUPPORTED, "batch * n_new * n_q_heads too large");
  return ok();
}

glance_status make_plan(const glance_attn_shape* s, Plan* out) {
  glance_status st = check_shape(s);
  if (st != GLANCE_OK) return st;
  glance::AttnParams p = {};
  p.batch = s->batch;
  p.n = s->n_new;
  p.hq = s->n_q_heads;
  p.hkv = s->n_kv_heads;
  p.group = s->n_q_heads / s->n_kv_heads;
  p.cap = s->ctx_capacity;
  p.d = s->head_dim;
  p.rows = p.n * p.group;
  const float scale = s->sm_scale > 0.f ? s->sm_scale : 1.0f / sqrtf((float)s->head_dim);
  p.scale_log2 = scale * 1.4426950408889634f;
  Plan pl;
  if (s->dtype == GLANCE_BF16) {
    // Row groups of at most seven 32-row tiles (seven computing waves and
    // the streaming wave), spread evenly; about one workgroup per compute
    // unit (256) over all piece slots, at least one slot per sequence.
    const int tiles = (p.rows + 31) / 32;
    p.row_groups = (tiles + 6) / 7;
    p.tiles_rg = (tiles + p.row_groups - 1) / p.row_groups;
    p.rows_rg = 32 * p.tiles_rg;
    const int per_g = 256 / (p.hkv * p.row_groups);
    p.slots_per_g = per_g > p.batch ? per_g : p.batch;
    p.min_tiles = 4;
    const size_t wslots = (size_t)p.slots_per_g * p.hkv * p.row_groups;
    pl.counter_bytes = round_up((size_t)p.batch * sizeof(int2), 256);
    pl.part_ml_bytes = round_up(wslots * p.rows_rg * sizeof(float2), 256);
    pl.part_o_bytes = round_up(wslots * p.rows_rg * p.d * sizeof(uint16_t), 256);  // fp16
  } else {
    p.row_groups = (p.rows + glance::kF32RowBlock - 1) / glance::kF32RowBlock;
    p.rows_pad = p.row_groups * glance::kF32RowBlock;
    p.split_keys = f32_split_keys(*s, p.row_groups);
    p.nsplit = p.cap > 0 ? (p.cap + p.split_keys - 1) / p.split_keys : 1;
    const size_t slots = (size_t)p.batch * p.hkv * p.nsplit * p.rows_pad;
    pl.counter_bytes = 0;
    pl.part_ml_bytes = round_up(slots * sizeof(float2), 256);
    pl.part_o_bytes = round_up(slots * p.d * sizeof(float), 256);
  }
  pl.total = pl.counter_bytes + pl.part_ml_bytes + pl.part_o_bytes;
  pl.p = p;
  *out = pl;
  return ok();
}

glance_status check_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return GLANCE_OK;
  return fail(GLANCE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

void take_events(hipEvent_t* a, hipEvent_t* b) {
  *a = g_ev_start;
  *b = g_ev_stop;
  g_ev_start = g_ev_stop = nullptr;
}

glance_status attn_common(bool tree, const glance_attn_shape* s, const void* q, const void* k_ctx,
                          const void* v_ctx, const void* k_new, const void* v_new,
                          const int32_t* ctx_lens, const int32_t* parents, void* out, float* lse,
                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
  Plan pl;
  glance_status st = make_plan(s, &pl);
  if (st != GLANCE_OK) return st;
  struct {
    const void* ptr;
    const char* name;
    bool need;
  } req[] = {{q, "q", true},           {k_new, "k_new", true},        {v_new, "v_new", true},
             {ctx_lens, "ctx_lens", true}, {out, "out", true},
             {k_ctx, "k_ctx", s->ctx_capacity > 0}, {v_ctx, "v_ctx", s->ctx_capacity > 0},
             {parents, "parents", tree}};
  for (auto& r : req) {
    if (r.need && !r.ptr) return fail(GLANCE_ERR_INVALID_ARG, "%s is NULL", r.name);
    if (r.ptr && !aligned16(r.ptr) && r.ptr != ctx_lens && r.ptr != parents)
      return fail(GLANCE_ERR_INVALID_ARG, "%s is not 16-byte aligned", r.name);
  }
  if ((reinterpret_cast<uintptr_t>(ctx_lens) & 3u) || (parents && (reinterpret_cast<uintptr_t>(parents) & 3u)))
    return fail(GLANCE_ERR_INVALID_ARG, "int32 arrays must be 4-byte aligned");
  if (lse && (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(GLANCE_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  if (!workspace) return fail(GLANCE_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(GLANCE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < pl.total)
    return fail(GLANCE_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes,
                pl.total);

  glance::AttnParams p = pl.p;
  p.q = q;
  p.k_ctx = k_ctx;
  p.v_ctx = v_ctx;
  p.k_new = k_new;
  p.v_new = v_new;
  p.ctx_lens = ctx_lens;
  p.parents = tree ? parents : nullptr;
  char* ws = static_cast<char*>(workspace);
  p.plan = pl.counter_bytes ? reinterpret_cast<int2*>(ws) : nullptr;
  p.part_ml = reinterpret_cast<float2*>(ws + pl.counter_bytes);
  p.part_o = reinterpret_cast<float*>(ws + pl.counter_bytes + pl.part_ml_bytes);
  p.out = out;
  p.lse = lse;
  hipEvent_t e0, e1;
  take_events(&e0, &e1);
  // the profiling events bracket the attention kernel (not the merge pass)
  hipError_t e = s->dtype == GLANCE_BF16 ? glance::launch_attn_bf16(p, tree, stream, e0, e1)
                                         : glance::launch_attn_f32(p, tree, stream, e0, e1);
  if ((st = check_hip(e, "attention kernel launch")) != GLANCE_OK) return st;
  e = s->dtype == GLANCE_BF16 ? glance::launch_attn_merge_pieces(p, stream)
                              : glance::launch_attn_merge(p, false, stream);
  return check_hip(e, "merge kernel launch");
}

struct AcceptPlan {
  int chunks, chunk_len;                // greedy acceptance (bandwidth-bound)
  int sample_chunks, sample_chunk_len;  // sampling walk (ALU-bound: more workgroups)
  size_t part_bytes, bytes;  // chunk words, then the root row's entropy chunks
};

glance_status accept_plan(int32_t batch, int32_t n_nodes, int32_t vocab, AcceptPlan* out) {
  if (batch < 1) return fail(GLANCE_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (n_nodes < 1 || n_nodes > 64)
    return fail(GLANCE_ERR_UNSUPPORTED, "n_nodes must be in 1..64 (got %d)", n_nodes);
  if (vocab < 1 || vocab > (1 << 30)) return fail(GLANCE_ERR_INVALID_ARG, "vocab must be in 1..2^30");
  const long long rows = (long long)batch * n_nodes;
  if (rows > (1LL << 40) / vocab) return fail(GLANCE_ERR_UNSUPPORTED, "logits too large");  // rows * vocab > 2^40
  // about 512 workgroups over the grid (two per CU), chunks of at least 8192 values
  const long long target = 512;
  long long chunks = (target + rows - 1) / rows;
  long long max_chunks = ((long long)vocab + 8191) / 8192;
  if (chunks > max_chunks) chunks = max_chunks;
  if (chunks < 1) chunks = 1;
  long long len = ((long long)vocab + chunks - 1) / chunks;
  len = (len + 7) / 8 * 8;
  chunks = ((long long)vocab + len - 1) / len;
  out->chunks = (int)chunks;
  out->chunk_len = (int)len;
  // sampling: about 2048 workgroups (eight waves a SIMD; measured best of
  // 512..4096 at 256 x 152064 bf16), chunks a multiple of 1024 tokens so that
  // only a row's last chunk has a ragged tail
  const long long s_target = 2048;
  long long s_chunks = (s_target + rows - 1) / rows;
  const long long s_max = ((long long)vocab + 4095) / 4096;
  if (s_chunks > s_max) s_chunks = s_max;
  if (s_chunks < 1) s_chunks = 1;
  long long s_len = ((long long)vocab + s_chunks - 1) / s_chunks;
  s_len = (s_len + 1023) / 1024 * 1024;
  s_chunks = ((long long)vocab + s_len - 1) / s_len;
  out->sample_chunks = (int)s_chunks;
  out->sample_chunk_len = (int)s_len;
  const long long max_chunks_any = chunks > s_chunks ? chunks : s_chunks;
  out->part_bytes = round_up((size_t)rows * max_chunks_any * sizeof(unsigned long long), 256);
  out->bytes = out->part_bytes + round_up((size_t)batch * chunks * sizeof(float4), 256);
  return ok();
}

struct TreePlan {
  glance::TreeParams p;  // sizes and workspace offsets; pointers filled per call
  size_t off_stats, off_sketch, off_thr, off_cand, off_ccount, off_lq, off_tok, bytes;
};

glance_status tree_plan(int32_t batch, int32_t horizon, int32_t vocab, int32_t budget, TreePlan* out) {
  if (batch < 1) return fail(GLANCE_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (horizon < 1) return fail(GLANCE_ERR_INVALID_ARG, "horizon must be >= 1 (got %d)", horizon);
  if (horizon > glance::kTreeMaxHorizon)
    return fail(GLANCE_ERR_UNSUPPORTED, "horizon must be <= %d (got %d)", glance::kTreeMaxHorizon, horizon);
  if (budget < 1) return fail(GLANCE_ERR_INVALID_ARG, "budget must be >= 1 (got %d)", budget);
  if (budget > glance::kTreeMaxBudget)
    return fail(GLANCE_ERR_UNSUPPORTED, "budget must be <= %d (got %d)", glance::kTreeMaxBudget, budget);
  if (vocab < 1 || vocab > (1 << 30)) return fail(GLANCE_ERR_INVALID_ARG, "vocab must be in 1..2^30");
  // the strings of length 1..horizon must number at least `budget`
  long long strings = 0, pw = 1;
  for (int l = 1; l <= horizon && strings < budget; ++l) {
    pw = pw * vocab > budget ? (long long)budget + 1 : pw * vocab;
    strings += pw;
  }
  if (strings < budget)
    return fail(GLANCE_ERR_INVALID_ARG, "budget %d exceeds the %lld strings of length <= %d over %d tokens",
                budget, strings, horizon, vocab);
  const long long rows = (long long)batch * horizon;
  if (rows > 65535) return fail(GLANCE_ERR_UNSUPPORTED, "batch * horizon must be <= 65535");
  if (rows * (long long)vocab > (1LL << 40)) return fail(GLANCE_ERR_UNSUPPORTED, "draft logits too large");
  glance::TreeParams p = {};
  p.batch = batch;
  p.horizon = horizon;
  p.vocab = vocab;
  p.budget = budget;
  p.k = budget < vocab ? budget : vocab;
  p.slices = (vocab + glance::kTreeSlice - 1) / glance::kTreeSlice;
  p.groups = 1;
  while ((long long)p.slices * p.groups < p.k && p.groups < 64) p.groups *= 2;
  // threshold buckets: four entries each when every bucket holds at least
  // four sketch entries, else one (the sketch has >= k entries)
  {
    const long long S = (long long)p.slices * p.groups;
    const int j = 4, nb = (p.k + j - 1) / j;
    if (S / nb >= j) {
      p.tau_buckets = nb;
      p.tau_rank = j;
    } else {
      p.tau_buckets = p.k;
      p.tau_rank = 1;
    }
  }
  p.wgs_per_row = (p.slices + glance::kTreeScanWaves * glance::kTreeSlicesPerWave - 1) /
                  (glance::kTreeScanWaves * glance::kTreeSlicesPerWave);
  TreePlan pl;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += round_up(bytes, 256);
    return at;
  };
  pl.off_stats = take((size_t)rows * p.slices * sizeof(float2));
  pl.off_sketch = take((size_t)rows * p.slices * p.groups * sizeof(float));
  pl.off_thr = take((size_t)rows * p.slices * sizeof(float));
  pl.off_cand = take((size_t)rows * p.slices * glance::kTreeSliceCap * sizeof(unsigned long long));
  pl.off_ccount = take((size_t)rows * p.slices * sizeof(int32_t));
  pl.off_lq = take((size_t)rows * 64 * sizeof(float));
  pl.off_tok = take((size_t)rows * 64 * sizeof(int32_t));
  pl.bytes = off;
  pl.p = p;
  *out = pl;
  return ok();
}

}  // namespace

extern "C" {

glance_status glance_block_draft_attn(const glance_attn_shape* s, const void* q, const void* k_ctx,
                                      const void* v_ctx, const void* k_new, const void* v_new,
                                      const int32_t* ctx_lens, void* out, float* lse,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return attn_common(false, s, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, nullptr, out, lse, workspace,
                     workspace_bytes, stream);
}

glance_status glance_tree_verify_attn(const glance_attn_shape* s, const void* q, const void* k_ctx,
                                      const void* v_ctx, const void* k_new, const void* v_new,
                                      const int32_t* ctx_lens, const int32_t* parents, void* out,
                                      float* lse, void* workspace, size_t workspace_bytes,
                                      hipStream_t stream) {
  return attn_common(true, s, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out, lse, workspace,
                     workspace_bytes, stream);
}

void bind_accept_workspace(glance::AcceptParams* p, const AcceptPlan& pl, void* workspace) {
  p->part = static_cast<unsigned long long*>(workspace);
  p->ent_part = reinterpret_cast<float4*>(static_cast<char*>(workspace) + pl.part_bytes);
}

// Host checks and parameters shared by the greedy and the sampling
// acceptance; `rows_name` names the per-row output in error messages.
glance_status accept_setup(int32_t batch, int32_t n_nodes, int32_t vocab, glance_dtype logits_dtype,
                           const void* logits, const int32_t* parents, const int32_t* tokens,
                           int32_t* rows_out, const char* rows_name, int32_t* accept_len,
                           int32_t* accept_path, int32_t path_stride, int32_t* next_root, void* workspace,
                           size_t workspace_bytes, AcceptPlan* pl, glance::AcceptParams* p) {
  glance_status st = accept_plan(batch, n_nodes, vocab, pl);
  if (st != GLANCE_OK) return st;
  if (!dtype_ok(logits_dtype)) return fail(GLANCE_ERR_UNSUPPORTED, "logits dtype must be GLANCE_F32 or GLANCE_BF16");
  if (path_stride < 1) return fail(GLANCE_ERR_INVALID_ARG, "path_stride must be >= 1");
  struct {
    const void* ptr;
    const char* name;
  } req[] = {{logits, "logits"},         {parents, "parents"},         {tokens, "tokens"},
             {rows_out, rows_name},      {accept_len, "accept_len"}, {accept_path, "accept_path"},
             {next_root, "next_root"}};
  for (auto& r : req) {
    if (!r.ptr) return fail(GLANCE_ERR_INVALID_ARG, "%s is NULL", r.name);
    if (reinterpret_cast<uintptr_t>(r.ptr) & 3u) return fail(GLANCE_ERR_INVALID_ARG, "%s is not 4-byte aligned", r.name);
  }
  if (logits_dtype == GLANCE_BF16 && (reinterpret_cast<uintptr_t>(logits) & 1u))
    return fail(GLANCE_ERR_INVALID_ARG, "logits is not 2-byte aligned");
  if (!workspace) return fail(GLANCE_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(GLANCE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < pl->bytes)
    return fail(GLANCE_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes,
                pl->bytes);
  *p = glance::AcceptParams{};
  p->logits = logits;
  p->parents = parents;
  p->tokens = tokens;
  p->argmax_out = rows_out;
  p->accept_len = accept_len;
  p->accept_path = accept_path;
  p->next_root = next_root;
  bind_accept_workspace(p, *pl, workspace);
  p->batch = batch;
  p->n_nodes = n_nodes;
  p->vocab = vocab;
  p->path_stride = path_stride;
  return ok();
}

namespace {
glance_status greedy_accept(int32_t batch, int32_t n_nodes, int32_t vocab, glance_dtype logits_dtype,
                            const void* logits, const int32_t* parents, const int32_t* tokens,
                            int32_t* argmax_out, int32_t* accept_len, int32_t* accept_path, int32_t path_stride,
                            int32_t* next_root, float* root_entropy, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  AcceptPlan pl;
  glance::AcceptParams p;
  glance_status st = accept_setup(batch, n_nodes, vocab, logits_dtype, logits, parents, tokens, argmax_out,
                                  "argmax_out", accept_len, accept_path, path_stride, next_root, workspace,
                                  workspace_bytes, &pl, &p);
  if (st != GLANCE_OK) return st;
  if (root_entropy && (reinterpret_cast<uintptr_t>(root_entropy) & 3u))
    return fail(GLANCE_ERR_INVALID_ARG, "root_entropy is not 4-byte aligned");
  p.root_entropy = root_entropy;
  p.chunks = pl.chunks;
  p.chunk_len = pl.chunk_len;
  hipEvent_t e0, e1;
  take_events(&e0, &e1);
  return check_hip(glance::launch_accept(p, logits_dtype == GLANCE_BF16, stream, e0, e1),
                   "accept kernel launch");
}
}  // namespace

glance_status glance_greedy_accept(int32_t batch, int32_t n_nodes, int32_t vocab,
                                   glance_dtype logits_dtype, const void* logits,
                                   const int32_t* parents, const int32_t* tokens,
                                   int32_t* argmax_out, int32_t* accept_len, int32_t* accept_path,
                                   int32_t path_stride, int32_t* next_root,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return greedy_accept(batch, n_nodes, vocab, logits_dtype, logits, parents, tokens, argmax_out, accept_len,
                       accept_path, path_stride, next_root, nullptr, workspace, workspace_bytes, stream);
}

glance_status glance_greedy_accept_noalloc(int32_t batch, int32_t n_nodes, int32_t vocab,
                                           glance_dtype logits_dtype, const void* logits,
                                           const int32_t* parents, const int32_t* tokens,
                                           int32_t* argmax_out, int32_t* accept_len, int32_t* accept_path,
                                           int32_t path_stride, int32_t* next_root, hipStream_t stream) {
  AcceptPlan pl;
  glance_status st = accept_plan(batch, n_nodes, vocab, &pl);
  if (st != GLANCE_OK) return st;
  const size_t cap = glance::noalloc_scratch_bytes();
  if (pl.bytes > cap)
    return fail(GLANCE_ERR_UNSUPPORTED,
                "batch %d x n_nodes %d x vocab %d needs %zu bytes of scratch; the static buffer holds %zu",
                batch, n_nodes, vocab, pl.bytes, cap);
  // every host check first, against an aligned placeholder of the right size
  glance::AcceptParams p;
  st = accept_setup(batch, n_nodes, vocab, logits_dtype, logits, parents, tokens, argmax_out, "argmax_out",
                    accept_len, accept_path, path_stride, next_root, reinterpret_cast<void*>(uintptr_t(256)),
                    pl.bytes, &pl, &p);
  if (st != GLANCE_OK) return st;
  void* ws = nullptr;
  if ((st = check_hip(glance::noalloc_scratch(&ws), "scratch address lookup")) != GLANCE_OK) return st;
  bind_accept_workspace(&p, pl, ws);
  p.chunks = pl.chunks;
  p.chunk_len = pl.chunk_len;
  hipEvent_t e0, e1;
  take_events(&e0, &e1);
  return check_hip(glance::launch_accept(p, logits_dtype == GLANCE_BF16, stream, e0, e1),
                   "accept kernel launch");
}

glance_status glance_greedy_accept_entropy(int32_t batch, int32_t n_nodes, int32_t vocab,
                                           glance_dtype logits_dtype, const void* logits,
                                           const int32_t* parents, const int32_t* tokens,
                                           int32_t* argmax_out, int32_t* accept_len, int32_t* accept_path,
                                           int32_t path_stride, int32_t* next_root, float* root_entropy,
                                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!root_entropy) return fail(GLANCE_ERR_INVALID_ARG, "root_entropy is NULL");
  return greedy_accept(batch, n_nodes, vocab, logits_dtype, logits, parents, tokens, argmax_out, accept_len,
                       accept_path, path_stride, next_root, root_entropy, workspace, workspace_bytes, stream);
}

glance_status glance_sample_accept(int32_t batch, int32_t n_nodes, int32_t vocab,
                                   glance_dtype logits_dtype, const void* logits,
                                   const int32_t* parents, const int32_t* tokens, float temperature,
                                   uint64_t seed, uint32_t round, uint32_t* round_counter, int32_t* draws_out,
                                   int32_t* accept_len, int32_t* accept_path, int32_t path_stride,
                                   int32_t* next_root, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  AcceptPlan pl;
  glance::AcceptParams p;
  glance_status st = accept_setup(batch, n_nodes, vocab, logits_dtype, logits, parents, tokens, draws_out,
                                  "draws_out", accept_len, accept_path, path_stride, next_root, workspace,
                                  workspace_bytes, &pl, &p);
  if (st != GLANCE_OK) return st;
  if (!(temperature >= FLT_MIN) || !(temperature <= FLT_MAX))
    return fail(GLANCE_ERR_INVALID_ARG, "temperature must be a finite normal float > 0 (got %g)",
                (double)temperature);
  p.chunks = pl.sample_chunks;
  p.chunk_len = pl.sample_chunk_len;
  p.temperature = temperature;
  p.inv_temperature = 1.0f / temperature;
  p.seed_lo = (unsigned)(seed & 0xffffffffu);
  p.seed_hi = (unsigned)(seed >> 32);
  if (round_counter && (reinterpret_cast<uintptr_t>(round_counter) & 3u))
    return fail(GLANCE_ERR_INVALID_ARG, "round_counter is not 4-byte aligned");
  p.round = round;
  p.round_counter = round_counter;
  hipEvent_t e0, e1;
  take_events(&e0, &e1);
  return check_hip(glance::launch_sample(p, logits_dtype == GLANCE_BF16, stream, e0, e1),
                   "sample kernel launch");
}

glance_status glance_build_tree(int32_t batch, int32_t horizon, int32_t vocab, int32_t budget,
                                glance_dtype logits_dtype, const void* draft_logits, int64_t seq_stride,
                                const int32_t* roots, int32_t* parents, int32_t* tokens, float* scores,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
  TreePlan pl;
  glance_status st = tree_plan(batch, horizon, vocab, budget, &pl);
  if (st != GLANCE_OK) return st;
  if (!dtype_ok(logits_dtype))
    return fail(GLANCE_ERR_UNSUPPORTED, "draft logits dtype must be GLANCE_F32 or GLANCE_BF16");
  if (seq_stride < (int64_t)horizon * vocab)
    return fail(GLANCE_ERR_INVALID_ARG, "seq_stride (%lld) must be >= horizon * vocab (%lld)",
                (long long)seq_stride, (long long)horizon * vocab);
  const size_t esz = logits_dtype == GLANCE_BF16 ? 2 : 4;
  if (!draft_logits) return fail(GLANCE_ERR_INVALID_ARG, "draft_logits is NULL");
  if (reinterpret_cast<uintptr_t>(draft_logits) & (esz - 1))
    return fail(GLANCE_ERR_INVALID_ARG, "draft_logits is not %zu-byte aligned", esz);
  struct {
    const void* ptr;
    const char* name;
  } req[] = {{roots, "roots"}, {parents, "parents"}, {tokens, "tokens"}};
  for (auto& r : req) {
    if (!r.ptr) return fail(GLANCE_ERR_INVALID_ARG, "%s is NULL", r.name);
    if (reinterpret_cast<uintptr_t>(r.ptr) & 3u) return fail(GLANCE_ERR_INVALID_ARG, "%s is not 4-byte aligned", r.name);
  }
  if (scores && (reinterpret_cast<uintptr_t>(scores) & 3u))
    return fail(GLANCE_ERR_INVALID_ARG, "scores is not 4-byte aligned");
  if (!workspace) return fail(GLANCE_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(GLANCE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < pl.bytes)
    return fail(GLANCE_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes,
                pl.bytes);
  glance::TreeParams p = pl.p;
  char* ws = static_cast<char*>(workspace);
  p.logits = draft_logits;
  p.seq_stride = seq_stride;
  p.roots = roots;
  p.parents = parents;
  p.tokens = tokens;
  p.scores = scores;
  p.stats = reinterpret_cast<float2*>(ws + pl.off_stats);
  p.sketch = reinterpret_cast<float*>(ws + pl.off_sketch);
  p.thr = reinterpret_cast<float*>(ws + pl.off_thr);
  p.cand = reinterpret_cast<unsigned long long*>(ws + pl.off_cand);
  p.lq = reinterpret_cast<float*>(ws + pl.off_lq);
  p.tok = reinterpret_cast<int32_t*>(ws + pl.off_tok);
  p.ccount = reinterpret_cast<int32_t*>(ws + pl.off_ccount);
  p.vec = (reinterpret_cast<uintptr_t>(draft_logits) & 15u) == 0 && ((size_t)vocab * esz) % 16 == 0 &&
          ((size_t)seq_stride * esz) % 16 == 0;
  hipEvent_t e0, e1;
  take_events(&e0, &e1);
  return check_hip(glance::launch_tree(p, logits_dtype == GLANCE_BF16, stream, e0, e1),
                   "tree builder kernel launch");
}

size_t glance_tree_workspace_size(int32_t batch, int32_t horizon, int32_t vocab, int32_t budget) {
  TreePlan pl;
  if (tree_plan(batch, horizon, vocab, budget, &pl) != GLANCE_OK) return 0;
  return pl.bytes;
}

glance_status glance_commit_path(int32_t batch, int32_t n_nodes, int32_t n_kv_heads, int32_t head_dim,
                                 int32_t ctx_capacity, glance_dtype dtype, const void* k_new,
                                 const void* v_new, const int32_t* accept_len, const int32_t* accept_path,
                                 int32_t path_stride, void* k_ctx, void* v_ctx, int32_t* ctx_lens,
                                 hipStream_t stream) {
  if (batch < 1) return fail(GLANCE_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (n_nodes < 1 || n_nodes > 64)
    return fail(GLANCE_ERR_UNSUPPORTED, "n_nodes must be in 1..64 (got %d)", n_nodes);
  if (n_kv_heads < 1) return fail(GLANCE_ERR_INVALID_ARG, "n_kv_heads must be >= 1");
  if (head_dim < 1 || head_dim > 1024) return fail(GLANCE_ERR_UNSUPPORTED, "head_dim must be in 1..1024");
  if (ctx_capacity < 1) return fail(GLANCE_ERR_INVALID_ARG, "ctx_capacity must be >= 1");
  if (path_stride < 1) return fail(GLANCE_ERR_INVALID_ARG, "path_stride must be >= 1");
  if (!dtype_ok(dtype))
    return fail(GLANCE_ERR_UNSUPPORTED, "dtype must be GLANCE_F32 or GLANCE_BF16");
  // per-sequence copy index arithmetic stays in 32 bits
  if ((long long)64 * n_kv_heads * head_dim * 2 > 0x7fffffffLL)
    return fail(GLANCE_ERR_UNSUPPORTED, "n_kv_heads * head_dim too large");
  const size_t esz = dtype == GLANCE_BF16 ? 2 : 4;
  struct {
    const void* ptr;
    const char* name;
    size_t align;
  } req[] = {{k_new, "k_new", esz},          {v_new, "v_new", esz},           {k_ctx, "k_ctx", esz},
             {v_ctx, "v_ctx", esz},          {accept_len, "accept_len", 4}, {accept_path, "accept_path", 4},
             {ctx_lens, "ctx_lens", 4}};
  for (auto& r : req) {
    if (!r.ptr) return fail(GLANCE_ERR_INVALID_ARG, "%s is NULL", r.name);
    if (reinterpret_cast<uintptr_t>(r.ptr) & (r.align - 1))
      return fail(GLANCE_ERR_INVALID_ARG, "%s is not %zu-byte aligned", r.name, r.align);
  }
  glance::CommitParams p = {};
  p.k_new = k_new;
  p.v_new = v_new;
  p.accept_len = accept_len;
  p.accept_path = accept_path;
  p.k_ctx = k_ctx;
  p.v_ctx = v_ctx;
  p.ctx_lens = ctx_lens;
  p.batch = batch;
  p.n = n_nodes;
  p.hkv = n_kv_heads;
  p.d = head_dim;
  p.cap = ctx_capacity;
  p.path_stride = path_stride;
  p.esz = (int)esz;
  p.vec = ((size_t)head_dim * esz) % 16 == 0 && aligned16(k_new) && aligned16(v_new) && aligned16(k_ctx) &&
          aligned16(v_ctx);
  hipEvent_t e0, e1;
  take_events(&e0, &e1);
  return check_hip(glance::launch_commit(p, stream, e0, e1), "commit kernel launch");
}

size_t glance_attn_workspace_size(const glance_attn_shape* s, int is_verify) {
  (void)is_verify;  // the draft and the verify of one shape share a plan
  Plan pl;
  if (make_plan(s, &pl) != GLANCE_OK) return 0;
  return pl.total;
}

size_t glance_accept_workspace_size(int32_t batch, int32_t n_nodes, int32_t vocab) {
  AcceptPlan pl;
  if (accept_plan(batch, n_nodes, vocab, &pl) != GLANCE_OK) return 0;
  return pl.bytes;
}

glance_status glance_validate_tree(int32_t n, const int32_t* parents, const int32_t* tokens,
                                   int32_t max_depth) {
  if (n < 1 || n > 64) return fail(GLANCE_ERR_INVALID_ARG, "tree size must be in 1..64 (got %d)", n);
  if (!parents) return fail(GLANCE_ERR_INVALID_ARG, "parents is NULL");
  if (parents[0] != -1) return fail(GLANCE_ERR_INVALID_ARG, "parents[0] must be -1 (got %d)", parents[0]);
  int depth[64];
  depth[0] = 0;
  for (int i = 1; i < n; ++i) {
    if (parents[i] < 0 || parents[i] >= i)
      return fail(GLANCE_ERR_INVALID_ARG, "parents[%d] = %d is not in [0, %d)", i, parents[i], i);
    depth[i] = depth[parents[i]] + 1;
    if (max_depth >= 0 && depth[i] > max_depth)
      return fail(GLANCE_ERR_INVALID_ARG, "node %d has depth %d > %d", i, depth[i], max_depth);
  }
  if (tokens) {
    for (int i = 1; i < n; ++i)
      for (int j = 1; j < i; ++j)
        if (parents[j] == parents[i] && tokens[j] == tokens[i])
          return fail(GLANCE_ERR_INVALID_ARG, "siblings %d and %d carry the same token %d", j, i, tokens[i]);
  }
  return ok();
}

const char* glance_status_string(glance_status status) {
  switch (status) {
    case GLANCE_OK: return "ok";
    case GLANCE_ERR_INVALID_ARG: return "invalid argument";
    case GLANCE_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case GLANCE_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case GLANCE_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* glance_last_error(void) { return g_last_error.c_str(); }

glance_status glance_set_kernel_events(void* start_event, void* stop_event) {
  if ((start_event == nullptr) != (stop_event == nullptr))
    return fail(GLANCE_ERR_INVALID_ARG, "pass both events or neither");
  g_ev_start = static_cast<hipEvent_t>(start_event);
  g_ev_stop = static_cast<hipEvent_t>(stop_event);
  return ok();
}

int32_t glance_version(void) { return 300; }

}  // extern "C"
