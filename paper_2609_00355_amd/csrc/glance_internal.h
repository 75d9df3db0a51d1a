// Internal interface between the C-ABI host layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace glance {

// Keys per LDS tile and waves per workgroup of the attention kernels.
constexpr int kKeyTile = 64;
constexpr int kWaves = 4;
// Rows per workgroup of the fp32 attention kernel (kWaves waves x 8 rows).
constexpr int kF32RowsPerWave = 8;
constexpr int kF32RowBlock = kWaves * kF32RowsPerWave;

// Everything a split-KV attention launch needs.  Layouts:
//   q      [batch][n][hq][d]         k_ctx/v_ctx [batch][hkv][cap][d]
//   k_new  [batch][n][hkv][d]        parents [batch][n]
//   part_o  fp32 kernel: [batch][hkv][nsplit][rows_pad][d] f32 (unnormalised partial output)
//           bf16 kernel: [slot * row_groups + rg][tiles_rg][d / 8][64 lanes] f16x4 (MFMA layout;
//           each row's O / sum scaled by 2^-e)
//   part_ml fp32 kernel: [batch][hkv][nsplit][rows_pad] f32x2 (running max * scale*log2e, sum)
//           bf16 kernel: [slot * row_groups + rg][rows_rg] f32x2 (max * scale*log2e + log2 sum + e, 2^-e)
//   out    [batch][n][hq][d]         lse [batch][n][hq]
// Row r of a (sequence, KV head) problem is new row r / group of query head
// g * group + r % group.
struct AttnParams {
  const void* q;
  const void* k_ctx;
  const void* v_ctx;
  const void* k_new;
  const void* v_new;
  const int32_t* ctx_lens;
  const int32_t* parents;  // null for the block draft
  float* part_o;
  float2* part_ml;
  void* out;
  float* lse;
  int batch, n, hq, hkv, group, cap, d;
  int rows;       // n * group
  int rows_pad;   // rows rounded up to the kernel's row block (fp32 kernel)
  int row_groups; // workgroups sharing one run of key tiles
  int nsplit;     // split slots per (sequence, KV head) = ceil(cap / split_keys), >= 1 (fp32 kernel)
  int split_keys; // context keys per split, multiple of kKeyTile (fp32 kernel)
  float scale_log2;  // sm_scale * log2(e)
  // bf16 kernel: pieces planned on the device from ctx_lens (see attn_bf16.hip)
  int slots_per_g;  // piece slots per KV head (>= batch)
  int min_tiles;    // smallest piece, in 64-key tiles
  int tiles_rg;     // 32-row tiles per row group (= computing waves, 1..7)
  int rows_rg;      // 32 * tiles_rg
  int2* plan;       // [batch] (pieces, first piece slot) of each sequence, for the merge pass
};

struct AcceptParams {
  const void* logits;
  const int32_t* parents;
  const int32_t* tokens;
  int32_t* argmax_out;
  int32_t* accept_len;
  int32_t* accept_path;
  int32_t* next_root;
  float* root_entropy;       // [batch] or null: entropy of each sequence's row 0
  unsigned long long* part;  // [batch * n_nodes][chunks] packed (key, ~index)
  float4* ent_part;          // [batch][chunks] (chunk max m, sum e^(z-m), sum e^(z-m) (z-m), 0)
  int batch, n_nodes, vocab, path_stride;
  int chunks, chunk_len;     // chunk_len is a multiple of 8
  // sampling walk only: the row draws are argmax(z / temperature + Gumbel)
  float temperature, inv_temperature;
  unsigned seed_lo, seed_hi, round;
  unsigned* round_counter;   // or null: added to round, then advanced by the walk
};

// Draft tree builder.  Limits: budget N <= kTreeMaxBudget strings below the
// root, horizon L <= kTreeMaxHorizon offsets (five 6-bit ranks per word, three
// words), K = min(N, vocab) ranked tokens kept per offset.
constexpr int kTreeMaxBudget = 63;
constexpr int kTreeMaxHorizon = 15;
constexpr int kTreeSlice = 1024;   // values per slice (one wave-wide load of 16 per lane)
constexpr int kTreeSlicesPerWave = 1;
constexpr int kTreeScanWaves = 4;   // waves per tree_scan workgroup
constexpr int kTreeSliceCap = 64;  // candidate slots per slice before it is re-read
constexpr int kTreeCap = 2048;     // candidates per row ranked by counting

// Layouts (row = sequence * L + offset - 1):
//   logits  sequence b, offset j (1..L) at logits + b*seq_stride + (j-1)*vocab
//   stats   [rows][slices] (max, sum exp(x - max)) of each 1024-value slice
//   sketch  [rows][slices * groups] maxima of disjoint lane groups
//   thr     [rows][slices] each slice's own candidate threshold
//   cand    [rows][slices][kTreeSliceCap] packed (order key, ~index) of the
//           slice's values >= thr; ccount [rows][slices] their number
//   lq, tok [rows][64] the row's K best tokens in rank order: tok[r] the token
//           of rank r, lq[r] the log q of rank r + 1 (-inf past the K-th),
//           lq[63] the log q of rank 0
struct TreeParams {
  const void* logits;
  long long seq_stride;
  const int32_t* roots;
  int32_t* parents;
  int32_t* tokens;
  float* scores;
  float2* stats;
  float* sketch;
  float* thr;
  unsigned long long* cand;
  float* lq;
  int32_t* tok;
  int32_t* ccount;
  int batch, horizon, vocab, budget;
  int k;            // ranked tokens per offset, min(budget, vocab)
  int slices;       // ceil(vocab / kTreeSlice)
  int groups;       // sketch entries per slice, a power of two in 1..64
  int tau_buckets;  // B: threshold buckets over the sketch
  int tau_rank;     // j in 1..4: the bucket entry of rank j bounds the threshold; B * j >= k
  int wgs_per_row;  // ceil(slices / (kTreeScanWaves * kTreeSlicesPerWave))
  int vec;          // rows are 16-byte aligned: vector loads
};

// Commit of an accepted path: k_new/v_new [batch][n][hkv][d] rows of the path
// nodes into k_ctx/v_ctx [batch][hkv][cap][d] at ctx_lens[b] + i.
struct CommitParams {
  const void* k_new;
  const void* v_new;
  const int32_t* accept_len;
  const int32_t* accept_path;
  void* k_ctx;
  void* v_ctx;
  int32_t* ctx_lens;
  int batch, n, hkv, d, cap, path_stride;
  int esz;  // bytes per element, 2 or 4
  int vec;  // rows are 16-byte multiples and every pointer is 16-byte aligned
};

hipError_t launch_attn_bf16(const AttnParams& p, bool tree, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
hipError_t launch_attn_f32(const AttnParams& p, bool tree, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
hipError_t launch_attn_merge(const AttnParams& p, bool out_bf16, hipStream_t s);
hipError_t launch_attn_merge_pieces(const AttnParams& p, hipStream_t s);
hipError_t launch_accept(const AcceptParams& p, bool bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
hipError_t launch_sample(const AcceptParams& p, bool bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
hipError_t launch_tree(const TreeParams& p, bool bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
hipError_t launch_commit(const CommitParams& p, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);

// The static per-GPU scratch of the allocation-free entry points: its size,
// and the current device's copy (looked up once per device).
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(void** out);

}  // namespace glance
