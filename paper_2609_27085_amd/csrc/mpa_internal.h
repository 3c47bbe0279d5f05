// Internal plan structures shared by the host planner (mpa_api.cpp) and the
// kernels (mpa_kernels.hip).  Plans travel as kernel arguments, so a launch
// needs no host-to-device copy and no device allocation.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpa {

constexpr int kBlock = 16;            // tokens per cache block
constexpr int kWavesPerGroup = 4;     // waves per workgroup in every kernel
constexpr int kMaxPlanSeqs = 256;     // sequences per launch (kernel-argument plan)
constexpr int kMaxPrefillSeqs = 64;   // prefill chunks per launch (its plan carries more per chunk)
constexpr int kPrefillSplitTarget = 256;  // prefill workgroups a launch should at least have
constexpr int kPrefillMinSplitTiles = 8;  // smallest KV range of a prefill split, in 64-key tiles
constexpr int kPrefillRows = 64;      // (token, head) rows per generic prefill workgroup
constexpr int kFewKeys = 64;          // rows that see at most this many keys get the 16-bit P pass
constexpr int kPrefillRowsMfma = 256; // (token, head) rows per bf16 prefill workgroup (8 waves)

// Pointers and sizes common to the attention kernels.
struct AttnArgs {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const int32_t* block_tables;
  const int32_t* seq_lens;
  const int32_t* qsl;
  void* out;
  float* lse;        // may be null
  float* ws_o;       // [items][Hq][d] split partial accumulators
  float* ws_ml;      // [items][Hq][2] split partial (max, sum); max in log2 units
  int32_t hq, hkv, mb, nb;
  float scale_log2;  // softmax scale * log2(e) (* the key scale for fp8 caches)
  float v_scale;     // fp8 caches: the value scale (1 otherwise), applied to outputs and partials
  // Decode rows' appends folded into the decode kernel (null: none).  The
  // wave that reads a decode row's last split first writes the row's new K
  // and V ([T][Hkv][d], query row order) for its KV head into the cache.
  const void* k_new;
  const void* v_new;
  float inv_k_scale, inv_v_scale;  // fp8 caches: 1 / scale, rounded to f32 (1 otherwise)
};

// Decode work for up to kMaxPlanSeqs sequences: item k of this launch is
// split x = k - item_start[j] of sequence seq[j], where item_start[j] <= k <
// item_start[j+1]; it covers keys [x * split_tokens[j], (x + 1) *
// split_tokens[j]) (a multiple of the block size; the last split ends at the
// sequence's length).  Its partial results live at workspace slot
// item_base + k.
struct DecodePlan {
  int32_t n_seqs;
  int32_t item_base;
  int32_t seq[kMaxPlanSeqs];
  int32_t split_tokens[kMaxPlanSeqs];
  int32_t item_start[kMaxPlanSeqs + 1];
};

// Prefill work for up to kMaxPrefillSeqs sequences.  Work unit k of this
// launch belongs to chunk j with tile_start[j] <= k < tile_start[j+1]; with
// u = k - tile_start[j] it is query tile u / nsplit[j] and KV split
// u % nsplit[j] of sequence seq[j].  Split x of a chunk covers 64-key tiles
// [x * split_tiles[j], (x + 1) * split_tiles[j]), the last split everything
// from there to the end; all splits but the last lie inside the cached
// prefix.  A chunk with nsplit > 1 writes per-split partial results for its
// token i and split x to workspace slot item_base[j] + x * C + i, and the
// merge launch combines them (grid.x runs over row_start, the chunks' token
// counts summed over split chunks only).
struct PrefillPlan {
  int32_t n_seqs;
  int32_t q_tile;    // query tokens per tile = rows per workgroup / G
  int32_t seq[kMaxPrefillSeqs];
  int32_t tile_start[kMaxPrefillSeqs + 1];
  int32_t nsplit[kMaxPrefillSeqs];
  int32_t split_tiles[kMaxPrefillSeqs];
  int32_t item_base[kMaxPrefillSeqs];
  int32_t row_start[kMaxPrefillSeqs + 1];
};

struct AppendArgs {
  const void* k_new;
  const void* v_new;
  void* k_cache;
  void* v_cache;
  const int32_t* block_tables;
  int32_t hkv, mb, nb;
  float inv_k_scale, inv_v_scale;  // fp8 caches: 1 / scale, rounded to f32 (1 otherwise)
};

// The rotary embedding applied by the rope append: query rows (in place,
// [T][Hq][d]) and the angle table cos_sin[pos][half][2] (cos, sin).
struct RopeArgs {
  void* q;
  const float* cos_sin;
  int32_t hq, half;
};

// Append work for up to kMaxPlanSeqs sequences: token k of this launch is new
// token (k - tok_start[j]) of sequence seq[j]; that token is query row
// row0[j] + (k - tok_start[j]) at position pos0[j] + (k - tok_start[j]).
struct AppendPlan {
  int32_t n_seqs;
  int32_t unit;  // 1 when every sequence of the plan adds exactly one token

  int32_t seq[kMaxPlanSeqs];
  int32_t row0[kMaxPlanSeqs];
  int32_t pos0[kMaxPlanSeqs];
  int32_t tok_start[kMaxPlanSeqs + 1];
};

// Append work for up to kMaxPrefillSeqs sequences that add several tokens,
// by cache block: unit u of this launch is the
// (u - unit_start[j])-th cache block touched by the new tokens of sequence
// seq[j].  Those tokens are query rows row0[j] .. row0[j] + ntok[j] - 1 at
// positions pos0[j] .. pos0[j] + ntok[j] - 1.
struct AppendBlockPlan {
  int32_t n_seqs;
  int32_t seq[kMaxPrefillSeqs];
  int32_t row0[kMaxPrefillSeqs];
  int32_t pos0[kMaxPrefillSeqs];
  int32_t ntok[kMaxPrefillSeqs];
  int32_t unit_start[kMaxPrefillSeqs + 1];
};

// Launchers (mpa_kernels.hip).  dtype: 0 = bf16, 1 = f32, 2 = fp8 cache.  Return the HIP
// error of the launch.
hipError_t launch_append(const AppendArgs& a, const AppendPlan& p, int dtype, int head_dim, hipStream_t stream);
// The same bits for multi-token sequences, one wave per (cache block, KV head).
hipError_t launch_append_blocks(const AppendArgs& a, const AppendBlockPlan& p, int dtype, int head_dim,
                                hipStream_t stream);
hipError_t launch_rope_append(const AppendArgs& a, const AppendPlan& p, const RopeArgs& r, int dtype, int head_dim,
                              hipStream_t stream);
// Decode waves the current device holds at once (2048 without a device).
int decode_wave_slots(int dtype, int head_dim);
hipError_t launch_decode(const AttnArgs& a, const DecodePlan& p, int n_items, int dtype, int head_dim,
                         hipStream_t stream);
hipError_t launch_merge(const AttnArgs& a, const DecodePlan& p, int dtype, int head_dim, hipStream_t stream);
hipError_t launch_prefill(const AttnArgs& a, const PrefillPlan& p, int n_tiles, int dtype, int head_dim,
                          hipStream_t stream);
// The generic (16 rows per wave) prefill kernel for any dtype; in bf16 it
// recomputes the rows of a chunk that see at most 64 keys, after the MFMA
// kernel, with the probabilities carried to about 16 bits.
// Combines the KV-split partial results of the plan's split chunks.
hipError_t launch_prefill_merge(const AttnArgs& a, const PrefillPlan& p, int dtype, int head_dim,
                                hipStream_t stream);

}  // namespace mpa
