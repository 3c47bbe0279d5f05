// C ABI of the mixed paged-attention library: host-side validation, the
// varlen planner (decode rows -> split-K work items, prefill chunks -> query
// tiles) and the launch sequence.  Every check runs before the first launch.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <functional>
#include <mutex>
#include <queue>
#include <unordered_set>
#include <vector>

#include "mpa.h"
#include "mpa_internal.h"

namespace {

using mpa::kBlock;
constexpr int kMaskWords = 8;  // CU-mask words: devices of up to 256 CUs

struct Batch {
  std::vector<int> decode;   // sequence ids with q_len == 1
  std::vector<int> prefill;  // sequence ids with q_len > 1
  long decode_tokens = 0;    // sum of KV lengths of decode rows
};

int check_shape(const mpa_shape* sh) {
  if (!sh) return MPA_ERR_INVALID;
  if (sh->num_seqs < 0 || sh->num_q_heads <= 0 || sh->num_kv_heads <= 0 || sh->num_blocks < 0 ||
      sh->max_blocks_per_seq < 0 || sh->total_q_tokens < 0 || !isfinite(sh->scale) || !(sh->scale > 0.f))
    return MPA_ERR_INVALID;
  if (sh->dtype != MPA_BF16 && sh->dtype != MPA_F32 && sh->dtype != MPA_FP8) return MPA_ERR_UNSUPPORTED;
  if (sh->dtype == MPA_FP8 && !(isfinite(sh->k_scale) && sh->k_scale > 0.f && isfinite(sh->v_scale) &&
                                sh->v_scale > 0.f))
    return MPA_ERR_INVALID;
  if (sh->head_dim != 64 && sh->head_dim != 128) return MPA_ERR_UNSUPPORTED;
  if (sh->block_size != kBlock) return MPA_ERR_UNSUPPORTED;
  if (sh->num_q_heads % sh->num_kv_heads != 0) return MPA_ERR_UNSUPPORTED;
  if (sh->num_q_heads / sh->num_kv_heads > 16) return MPA_ERR_UNSUPPORTED;
  return MPA_OK;
}

// The MFMA prefill launch's work units (query tiles x KV heads) over the
// chunks, and the most KV splits any chunk's prefix allows.
void prefill_units(const mpa_shape* sh, const std::vector<int>& prefill, const int32_t* seq_lens,
                   const int32_t* qsl, long* units, int* most) {
  const int qt = mpa::kPrefillRowsMfma / (sh->num_q_heads / sh->num_kv_heads);
  *units = 0;
  *most = 1;
  for (int s : prefill) {
    const int C = qsl[s + 1] - qsl[s];
    *units += (long)(C + qt - 1) / qt * sh->num_kv_heads;
    *most = std::max(*most, std::min(1 + (seq_lens[s] - C) / 64 / mpa::kPrefillMinSplitTiles, 64));
  }
}

// Whether the planner leaves every prefill chunk of the batch whole (one KV
// split each): f32 chunks, and MFMA batches with at least two workgroups
// per CU or no prefix long enough to split, unless MPA_PREFILL_SPLITS
// overrides the choice.  prefill_splits() takes the same decision.
bool prefill_whole(const mpa_shape* sh, const std::vector<int>& prefill, const int32_t* seq_lens,
                   const int32_t* qsl) {
  if (sh->dtype == MPA_F32 || prefill.empty()) return true;
  if (const char* env = getenv("MPA_PREFILL_SPLITS")) {
    const int v = atoi(env);
    if (v >= 1 && v <= 64) return false;
  }
  long units;
  int most;
  prefill_units(sh, prefill, seq_lens, qsl, &units, &most);
  return units >= 2L * mpa::kPrefillSplitTarget || most == 1;
}

// Validates the host metadata and classifies the sequences.
int check_batch(const mpa_shape* sh, const int32_t* seq_lens, const int32_t* qsl, const int32_t* bt_host,
                bool append_only, Batch* b) {
  int rc = check_shape(sh);
  if (rc != MPA_OK) return rc;
  const int S = sh->num_seqs;
  if (S > 0 && (!seq_lens || !qsl)) return MPA_ERR_INVALID;
  if (S == 0) return sh->total_q_tokens == 0 ? MPA_OK : MPA_ERR_INVALID;
  if (qsl[0] != 0 || qsl[S] != sh->total_q_tokens) return MPA_ERR_INVALID;
  for (int s = 0; s < S; ++s) {
    const int ql = qsl[s + 1] - qsl[s];
    const int L = seq_lens[s];
    if (ql < 0 || L < 0 || ql > L) return MPA_ERR_INVALID;
    if (ql == 0) continue;
    if (sh->num_blocks == 0) return MPA_ERR_INVALID;  // nothing could hold its KV
    const long nblk = ((long)L + kBlock - 1) / kBlock;
    if (nblk > sh->max_blocks_per_seq) return MPA_ERR_INVALID;
    if (bt_host) {
      const long first = append_only ? (long)(L - ql) / kBlock : 0;
      for (long j = first; j < nblk; ++j) {
        const int32_t id = bt_host[(size_t)s * sh->max_blocks_per_seq + j];
        if (id < 0 || id >= sh->num_blocks) return MPA_ERR_INVALID;
      }
    }
    if (ql == 1) {
      b->decode.push_back(s);
      b->decode_tokens += L;
    } else {
      b->prefill.push_back(s);
    }
  }
  // The MFMA prefill kernel dispatches its work units from the plan's last
  // chunk backwards, each chunk from its longest query tile (the one that
  // sees all L keys).  With whole chunks ordered by L, the longest units go
  // first and the short ones fill the end of the launch.  A split chunk's
  // units are not ordered by length, so split batches keep batch order.
  if (sh->dtype != MPA_F32 && b->prefill.size() > 1 && prefill_whole(sh, b->prefill, seq_lens, qsl))
    std::stable_sort(b->prefill.begin(), b->prefill.end(), [&](int x, int y) { return seq_lens[x] < seq_lens[y]; });
  return MPA_OK;
}

// How a decode row of L keys is split at nominal split size S: into
// n = ceil(L / S) parts of equal size, rounded up to whole cache blocks, so
// that the waves of a launch stream about the same number of bytes (a fixed
// size S with a short remainder would leave the short waves idle while the
// full ones finish).  The last part ends at L; `parts` can be below n when
// the rounding makes the earlier parts cover L sooner.
struct RowSplit {
  int parts;
  int tokens;  // keys per part, a multiple of the block size
};

RowSplit row_split(int L, int S) {
  const int n = std::max(1, (L + S - 1) / S);
  const int per = (L + n - 1) / n;
  const int tokens = std::max(kBlock, (per + kBlock - 1) / kBlock * kBlock);
  return {std::max(1, (L + tokens - 1) / tokens), tokens};
}

// KV tokens per decode split.  Every (split, KV head) is one wave, and a
// wave's time is about proportional to its tokens plus a fixed start-up cost,
// so the step takes about ceil(waves / slots) * (split + overhead), where
// slots is the number of waves the device runs at once.  The split is the
// multiple of 16 in [128, 1024] that minimises that estimate (more, smaller
// splits fill the last round of waves; fewer, larger ones cut start-up and
// merge work).  MPA_SPLIT_TOKENS (a multiple of 16, at most 1024) overrides
// it for tuning sweeps.
int choose_split_uncached(const mpa_shape* sh, const Batch& b, const int32_t* seq_lens) {
  if (const char* env = getenv("MPA_SPLIT_TOKENS")) {
    const int v = atoi(env);
    if (v >= kBlock && v <= 1024 && v % kBlock == 0) return v;
  }
  if (b.decode.empty()) return 1024;
  const long slots = mpa::decode_wave_slots(sh->dtype, sh->head_dim);
  const long overhead = 64;
  long best_cost = -1;
  int best = 1024;
  for (int split = 128; split <= 1024; split += kBlock) {
    long items = 0;
    for (int s : b.decode) items += row_split(seq_lens[s], split).parts;
    const long waves = items * sh->num_kv_heads;
    const long cost = ((waves + slots - 1) / slots) * (split + overhead);
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best = split;
    }
  }
  return best;
}

// Per-thread memo of the last batch's two plan choices (the decode split
// and the prefill split count).  One step plans its batch several times --
// workspace sizing, the append, each attention half, the step model -- and
// the searches behind the choices cost more host time than the rest of the
// plan.  The key is everything the choices depend on: the shape's heads,
// head_dim and dtype, the exact seq_lens and query_start_loc, the device
// (its wave capacity) and the tuning overrides in the environment.
struct PlanMemo {
  int32_t key[7] = {-1, -1, -1, -1, -1, -1, -1};
  std::vector<int32_t> seq_lens, qsl;
  int split = 0;  // 0: not chosen yet
  int want = 0;
};

int env_int(const char* name) {
  const char* e = getenv(name);
  return e ? atoi(e) : -1;
}

PlanMemo& plan_memo(const mpa_shape* sh, const int32_t* seq_lens, const int32_t* qsl) {
  thread_local PlanMemo m;
  // an empty batch may come without metadata (check_batch accepts null
  // arrays when num_seqs is 0): its query_start_loc is {0}
  static const int32_t kEmptyQsl[1] = {0};
  if (sh->num_seqs == 0 && !qsl) qsl = kEmptyQsl;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) dev = -1;
  const int32_t key[7] = {sh->num_q_heads, sh->num_kv_heads, sh->head_dim, (int32_t)sh->dtype, dev,
                          env_int("MPA_SPLIT_TOKENS"), env_int("MPA_PREFILL_SPLITS")};
  const size_t n = (size_t)sh->num_seqs;
  if (memcmp(key, m.key, sizeof key) != 0 || m.seq_lens.size() != n || m.qsl.size() != n + 1 ||
      (n && memcmp(m.seq_lens.data(), seq_lens, n * sizeof(int32_t)) != 0) ||
      memcmp(m.qsl.data(), qsl, (n + 1) * sizeof(int32_t)) != 0) {
    memcpy(m.key, key, sizeof key);
    m.seq_lens.assign(seq_lens, seq_lens + n);
    m.qsl.assign(qsl, qsl + n + 1);
    m.split = m.want = 0;
  }
  return m;
}

int choose_split(const mpa_shape* sh, const Batch& b, const int32_t* seq_lens, const int32_t* qsl) {
  PlanMemo& m = plan_memo(sh, seq_lens, qsl);
  if (m.split == 0) m.split = choose_split_uncached(sh, b, seq_lens);
  return m.split;
}

long decode_items(const mpa_shape* sh, const Batch& b, const int32_t* seq_lens, int split) {
  (void)sh;
  long n = 0;
  for (int s : b.decode) n += row_split(seq_lens[s], split).parts;
  return n;
}

// Query tokens per prefill tile: 256 (token, head) rows for the MFMA kernel
// (bf16 and fp8 caches), 64 for the generic kernel (f32).
int q_tile(const mpa_shape* sh) {
  const int rows = sh->dtype == MPA_F32 ? mpa::kPrefillRows : mpa::kPrefillRowsMfma;
  return rows / (sh->num_q_heads / sh->num_kv_heads);
}

// Launch errors are read with hipGetLastError() after each launch.  That
// call also returns an error left behind by an earlier runtime call on this
// thread that nobody collected -- e.g. hipErrorNotReady from another
// library's stream or event query -- so it is cleared once, after
// validation, before this call's first launch.
void clear_stale_hip_error() { (void)hipGetLastError(); }

size_t workspace_bytes(const mpa_shape* sh, long items) {
  const size_t per = (size_t)sh->num_q_heads * (sh->head_dim + 2) * sizeof(float);
  return items * per;
}

// KV splits of the prefill chunks.  A chunk's query tiles times the KV heads
// are its workgroups, and each workgroup holds a whole CU.  With `want`
// splits, each chunk's cached prefix is divided among up to `want` parts of
// kPrefillMinSplitTiles 64-key tiles or more; the last split also takes the
// chunk's own keys (and the causal diagonal), so every split holds keys of
// every row.  bf16 and fp8 caches (the MFMA kernel); f32 chunks are not
// split.
struct PrefillSplit {
  int nsplit = 1;
  int tiles = 0;        // 64-key tiles of every split but the last
  long item_base = 0;   // first workspace slot of the chunk's partials
};

std::vector<PrefillSplit> split_layout(const Batch& b, const int32_t* seq_lens, const int32_t* qsl, int want,
                                       long first_item) {
  std::vector<PrefillSplit> out(b.prefill.size());
  long item = first_item;
  for (size_t k = 0; k < b.prefill.size(); ++k) {
    const int s = b.prefill[k];
    const int C = qsl[s + 1] - qsl[s];
    const int np = (seq_lens[s] - C) / 64;  // whole 64-key tiles of the prefix
    const int ct = (C + 63) / 64;
    const int n = std::min({want, 1 + np / mpa::kPrefillMinSplitTiles, 64});
    if (n < 2) continue;
    out[k].nsplit = n;
    out[k].tiles = std::min((np + ct + n - 1) / n, np / (n - 1));
    out[k].item_base = item;
    item += (long)n * C;
  }
  return out;
}

// Predicted device time of the prefill launches for a split layout: per
// launch (kMaxPrefillSeqs chunks), the makespan of its workgroups -- each
// wg_us + tile_us per 64-key tile -- dealt in launch order (the longest
// query tiles first) to `slots` slots that take the next workgroup when
// free; plus, when a chunk of the launch is split, the merge: merge_us +
// merge_row_us per partial (token, q head, split) row.
double prefill_time(const mpa_shape* sh, const Batch& b, const int32_t* seq_lens, const int32_t* qsl,
                    const std::vector<PrefillSplit>& sp, double wg_us, double tile_us, int slots, double merge_us,
                    double merge_row_us) {
  const int qt = q_tile(sh);
  double total = 0.0;
  std::vector<int> tiles;
  for (size_t c0 = 0; c0 < b.prefill.size(); c0 += mpa::kMaxPrefillSeqs) {
    const size_t c1 = std::min(b.prefill.size(), c0 + mpa::kMaxPrefillSeqs);
    tiles.clear();  // 64-key tiles of each work unit, in unit order
    double partial_rows = 0.0;
    for (size_t k = c0; k < c1; ++k) {
      const int s = b.prefill[k];
      const int C = qsl[s + 1] - qsl[s];
      const int P = seq_lens[s] - C;
      if (sp[k].nsplit > 1) partial_rows += (double)C * sh->num_q_heads * sp[k].nsplit;
      for (int q = 0; q < (C + qt - 1) / qt; ++q) {
        const int kend = P + std::min(q * qt + qt - 1, C - 1) + 1;
        const int all = (kend + 63) / 64;
        for (int x = 0; x < sp[k].nsplit; ++x)
          tiles.push_back(x == sp[k].nsplit - 1 ? all - x * sp[k].tiles : sp[k].tiles);
      }
    }
    std::priority_queue<double, std::vector<double>, std::greater<double>> free_at;
    for (int i = 0; i < slots; ++i) free_at.push(0.0);
    double makespan = 0.0;
    // blockIdx order: the last unit first, each unit once per KV head
    for (size_t u = tiles.size(); u-- > 0;)
      for (int g = 0; g < sh->num_kv_heads; ++g) {
        const double end = free_at.top() + wg_us + tile_us * tiles[u];
        free_at.pop();
        makespan = std::max(makespan, end);
        free_at.push(end);
      }
    total += makespan + (partial_rows > 0 ? merge_us + merge_row_us * partial_rows : 0.0);
  }
  return total;
}

// The planner's own figures for prefill_time (those of mpa_default_rates),
// fixed so that a batch always gets the same plan.
constexpr double kPlanWgUs = 18.0;
constexpr double kPlanTileUs = 1.85;
constexpr double kPlanMergeUs = 3.0;
constexpr double kPlanMergeRowUs = 1.6e-4;

// The split count.  A batch with at least two workgroups per CU is not
// split: its makespan is already close to its work over the CUs, and the
// partial results would cost more than they balance.  A smaller batch gets
// the split count (1, 2, ...) with the shortest predicted prefill time,
// the fewer splits on a tie; counts past the point where every chunk's
// prefix is cut as finely as allowed, or past 8 workgroups per CU, are not
// tried.  MPA_PREFILL_SPLITS (1..64) overrides the choice for tuning sweeps.
std::vector<PrefillSplit> prefill_splits(const mpa_shape* sh, const Batch& b, const int32_t* seq_lens,
                                         const int32_t* qsl, long first_item) {
  if (sh->dtype == MPA_F32 || b.prefill.empty()) return std::vector<PrefillSplit>(b.prefill.size());
  if (const char* env = getenv("MPA_PREFILL_SPLITS")) {
    const int v = atoi(env);
    if (v >= 1 && v <= 64) return split_layout(b, seq_lens, qsl, v, first_item);
  }
  if (prefill_whole(sh, b.prefill, seq_lens, qsl)) return std::vector<PrefillSplit>(b.prefill.size());
  long units;
  int most;  // the most splits any chunk can take
  prefill_units(sh, b.prefill, seq_lens, qsl, &units, &most);
  PlanMemo& m = plan_memo(sh, seq_lens, qsl);
  if (m.want == 0) {
    double best_t = -1.0;
    for (int want = 1; want <= most && (want == 1 || units * want <= 8L * mpa::kPrefillSplitTarget); ++want) {
      const double t = prefill_time(sh, b, seq_lens, qsl, split_layout(b, seq_lens, qsl, want, 0), kPlanWgUs,
                                    kPlanTileUs, mpa::kPrefillSplitTarget, kPlanMergeUs, kPlanMergeRowUs);
      if (best_t < 0 || t < best_t * (1.0 - 1e-9)) {
        best_t = t;
        m.want = want;
      }
    }
  }
  return split_layout(b, seq_lens, qsl, m.want, first_item);
}

long prefill_items(const std::vector<PrefillSplit>& sp, const Batch& b, const int32_t* qsl) {
  long n = 0;
  for (size_t k = 0; k < sp.size(); ++k)
    if (sp[k].nsplit > 1) n += (long)sp[k].nsplit * (qsl[b.prefill[k] + 1] - qsl[b.prefill[k]]);
  return n;
}

// MPA_DEBUG=1 (read per call): before an append, the cache slots it writes
// must be pairwise distinct, and none may hold a key that a sequence of the
// step reads (prefix blocks shared between sequences are read-only).  Needs
// the host copy of the block tables; without it the check cannot run and
// the call is rejected.  Costs a pass over every key of the step.
bool debug_checks() {
  const char* e = getenv("MPA_DEBUG");
  return e && e[0] == '1' && e[1] == '\0';
}

int check_append_slots(const mpa_shape* sh, const int32_t* seq_lens, const int32_t* qsl, const int32_t* bt) {
  if (!bt) return MPA_ERR_INVALID;
  std::unordered_set<int64_t> written;
  auto slot_of = [&](int s, int p) {
    return (int64_t)bt[(size_t)s * sh->max_blocks_per_seq + p / kBlock] * kBlock + p % kBlock;
  };
  for (int s = 0; s < sh->num_seqs; ++s) {
    const int ql = qsl[s + 1] - qsl[s];
    for (int p = seq_lens[s] - ql; p < seq_lens[s]; ++p)
      if (!written.insert(slot_of(s, p)).second) return MPA_ERR_INVALID;  // two tokens, one slot
  }
  for (int s = 0; s < sh->num_seqs; ++s) {
    const int ql = qsl[s + 1] - qsl[s];
    if (ql == 0) continue;
    for (int p = 0; p < seq_lens[s] - ql; ++p)
      if (written.count(slot_of(s, p))) return MPA_ERR_INVALID;  // overwrites a key that is read
  }
  return MPA_OK;
}

// The append launches (plain, or with the rotary embedding when rope is
// given): one wave per new token, up to kMaxPlanSeqs sequences per launch.
int run_append(const mpa_shape* shape, const void* k_new, const void* v_new, void* k_cache, void* v_cache,
               const int32_t* block_tables, const int32_t* seq_lens, const int32_t* query_start_loc,
               const int32_t* seq_lens_host, const int32_t* query_start_loc_host, const int32_t* block_tables_host,
               const mpa::RopeArgs* rope, void* stream, bool multi_only = false) {
  Batch b;
  int rc = check_batch(shape, seq_lens_host, query_start_loc_host, block_tables_host, true, &b);
  if (rc != MPA_OK) return rc;
  if (shape->total_q_tokens == 0) return MPA_OK;
  if (debug_checks()) {
    rc = check_append_slots(shape, seq_lens_host, query_start_loc_host, block_tables_host);
    if (rc != MPA_OK) return rc;
  }
  if (!k_new || !v_new || !k_cache || !v_cache || !block_tables || !seq_lens || !query_start_loc)
    return MPA_ERR_INVALID;
  mpa::AppendArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.block_tables = block_tables;
  a.hkv = shape->num_kv_heads;
  a.mb = shape->max_blocks_per_seq;
  a.nb = shape->num_blocks;
  a.inv_k_scale = shape->dtype == MPA_FP8 ? 1.f / shape->k_scale : 1.f;
  a.inv_v_scale = shape->dtype == MPA_FP8 ? 1.f / shape->v_scale : 1.f;
  (void)seq_lens;
  (void)query_start_loc;
  // single-token sequences one wave per token; with the rotary embedding
  // (which also rotates q, token by token) every sequence
  std::vector<int> seqs(b.decode);
  if (rope) seqs.insert(seqs.end(), b.prefill.begin(), b.prefill.end());
  if (multi_only) seqs.clear();  // the decode kernel appends the single-token rows
  clear_stale_hip_error();
  // multi-token sequences one wave per (cache block, KV head)
  if (!rope) {
    for (size_t c0 = 0; c0 < b.prefill.size(); c0 += mpa::kMaxPrefillSeqs) {
      mpa::AppendBlockPlan p;
      memset(&p, 0, sizeof(p));
      const size_t c1 = std::min(b.prefill.size(), c0 + mpa::kMaxPrefillSeqs);
      p.n_seqs = (int32_t)(c1 - c0);
      int acc = 0;
      for (size_t k = c0; k < c1; ++k) {
        const int s = b.prefill[k];
        const int ql = query_start_loc_host[s + 1] - query_start_loc_host[s];
        const int pos0 = seq_lens_host[s] - ql;
        p.seq[k - c0] = s;
        p.row0[k - c0] = query_start_loc_host[s];
        p.pos0[k - c0] = pos0;
        p.ntok[k - c0] = ql;
        p.unit_start[k - c0] = acc;
        acc += (pos0 + ql - 1) / kBlock - pos0 / kBlock + 1;
      }
      p.unit_start[c1 - c0] = acc;
      if (mpa::launch_append_blocks(a, p, shape->dtype, shape->head_dim, (hipStream_t)stream) != hipSuccess)
        return MPA_ERR_HIP;
    }
  }
  for (size_t c0 = 0; c0 < seqs.size(); c0 += mpa::kMaxPlanSeqs) {
    mpa::AppendPlan p;
    memset(&p, 0, sizeof(p));
    const size_t c1 = std::min(seqs.size(), c0 + mpa::kMaxPlanSeqs);
    p.n_seqs = (int32_t)(c1 - c0);
    int acc = 0;
    for (size_t k = c0; k < c1; ++k) {
      const int s = seqs[k];
      const int ql = query_start_loc_host[s + 1] - query_start_loc_host[s];
      p.seq[k - c0] = s;
      p.row0[k - c0] = query_start_loc_host[s];
      p.pos0[k - c0] = seq_lens_host[s] - ql;
      p.tok_start[k - c0] = acc;
      acc += ql;
    }
    p.tok_start[c1 - c0] = acc;
    p.unit = acc == (int)(c1 - c0) ? 1 : 0;
    hipError_t e = rope ? mpa::launch_rope_append(a, p, *rope, shape->dtype, shape->head_dim, (hipStream_t)stream)
                        : mpa::launch_append(a, p, shape->dtype, shape->head_dim, (hipStream_t)stream);
    if (e != hipSuccess) return MPA_ERR_HIP;
  }
  return MPA_OK;
}

}  // namespace

namespace {

// The step-time model (mpa_predict_step), shared with the mode planner.
mpa_step_time model_step(const mpa_shape* shape, const Batch& b, const int32_t* seq_lens_host,
                         const int32_t* qsl_host, const mpa_rates& r) {
  const double elem = 2.0;  // bf16
  const double row_bytes = (double)shape->num_kv_heads * shape->head_dim * elem;  // one token's K (or V)
  mpa_step_time t = {0.0, 0.0, 0.0, 0.0};

  // append, launch by launch as run_append issues them: every new token's K
  // and V read once and written once
  for (size_t c0 = 0; c0 < b.decode.size(); c0 += mpa::kMaxPlanSeqs) {
    const double tokens = (double)(std::min(b.decode.size(), c0 + mpa::kMaxPlanSeqs) - c0);
    t.append_us += r.append_fixed_us + 4.0 * row_bytes * tokens / (r.append_gbs * 1e3);
  }
  for (size_t c0 = 0; c0 < b.prefill.size(); c0 += mpa::kMaxPrefillSeqs) {
    double tokens = 0.0;
    for (size_t k = c0; k < std::min(b.prefill.size(), c0 + mpa::kMaxPrefillSeqs); ++k)
      tokens += qsl_host[b.prefill[k] + 1] - qsl_host[b.prefill[k]];
    t.append_us += std::max(r.append_block_us, 4.0 * row_bytes * tokens / (r.append_block_gbs * 1e3));
  }

  // decode, launch by launch as run_attention issues them
  const int split = choose_split(shape, b, seq_lens_host, qsl_host);
  const double head_bytes = 2.0 * shape->head_dim * elem;  // K + V of one token and KV head
  for (size_t c0 = 0; c0 < b.decode.size(); c0 += mpa::kMaxPlanSeqs) {
    const size_t c1 = std::min(b.decode.size(), c0 + mpa::kMaxPlanSeqs);
    double bytes = 0.0, wave = 0.0;
    bool split_any = false;
    for (size_t k = c0; k < c1; ++k) {
      const int L = seq_lens_host[b.decode[k]];
      bytes += (double)L * head_bytes * shape->num_kv_heads;
      wave = std::max(wave, (double)std::min(L, row_split(L, split).tokens) * head_bytes);
      split_any |= row_split(L, split).parts > 1;
    }
    t.decode_us += r.decode_fixed_us + std::max(bytes / (r.decode_gbs * 1e3), wave / (r.decode_wave_gbs * 1e3));
    if (split_any) t.decode_us += r.merge_us;
  }

  // prefill: each launch's workgroups, in launch order (longest query tiles
  // first), on prefill_slots slots that take the next workgroup when free
  const std::vector<PrefillSplit> psplit =
      prefill_splits(shape, b, seq_lens_host, qsl_host, decode_items(shape, b, seq_lens_host, split));
  t.prefill_us = prefill_time(shape, b, seq_lens_host, qsl_host, psplit, r.prefill_wg_us, r.prefill_tile_us,
                              r.prefill_slots, r.prefill_merge_us, r.prefill_merge_row_us);
  bool few = false;
  for (int s : b.prefill) few |= seq_lens_host[s] - (qsl_host[s + 1] - qsl_host[s]) < mpa::kFewKeys;
  if (few) t.prefill_us += r.prefill_fixup_us;
  t.step_us = t.append_us + t.decode_us + t.prefill_us;
  return t;
}

int check_model_inputs(const mpa_shape* shape, const int32_t* seq_lens_host, const int32_t* qsl_host,
                       const mpa_rates& r, Batch* b) {
  int rc = check_batch(shape, seq_lens_host, qsl_host, nullptr, false, b);
  if (rc != MPA_OK) return rc;
  if (shape->dtype != MPA_BF16) return MPA_ERR_UNSUPPORTED;
  if (!(r.append_gbs > 0) || !(r.append_block_gbs > 0) || !(r.decode_gbs > 0) || !(r.decode_wave_gbs > 0) ||
      r.prefill_slots <= 0)
    return MPA_ERR_INVALID;
  return MPA_OK;
}

}  // namespace

extern "C" {

const char* mpa_status_string(int status) {
  switch (status) {
    case MPA_OK: return "ok";
    case MPA_ERR_INVALID: return "invalid argument or batch metadata";
    case MPA_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case MPA_ERR_WORKSPACE: return "workspace missing, too small or not 16-byte aligned";
    case MPA_ERR_HIP: return "HIP launch error";
    case MPA_ERR_SCRATCH: return "batch needs more than the library's fixed scratch array (MPA_SCRATCH_BYTES)";
    default: return "unknown status";
  }
}

int mpa_get_plan_info(const mpa_shape* shape, const int32_t* seq_lens_host, const int32_t* qsl_host,
                      mpa_plan_info* info) {
  if (!info) return MPA_ERR_INVALID;
  Batch b;
  int rc = check_batch(shape, seq_lens_host, qsl_host, nullptr, false, &b);
  if (rc != MPA_OK) return rc;
  const int split = choose_split(shape, b, seq_lens_host, qsl_host);
  info->num_decode_seqs = (int32_t)b.decode.size();
  info->num_prefill_seqs = (int32_t)b.prefill.size();
  info->split_tokens = split;
  info->num_decode_items = (int32_t)decode_items(shape, b, seq_lens_host, split);
  long tiles = 0;
  const int qt = q_tile(shape);
  const std::vector<PrefillSplit> ps =
      prefill_splits(shape, b, seq_lens_host, qsl_host, decode_items(shape, b, seq_lens_host, split));
  int max_split = b.prefill.empty() ? 0 : 1;
  for (size_t k = 0; k < b.prefill.size(); ++k) {
    const int s = b.prefill[k];
    tiles += (long)(qsl_host[s + 1] - qsl_host[s] + qt - 1) / qt * ps[k].nsplit;
    max_split = std::max(max_split, ps[k].nsplit);
  }
  info->num_prefill_tiles = (int32_t)(tiles * shape->num_kv_heads);
  info->prefill_max_splits = max_split;
  info->decode_launches = (int32_t)((b.decode.size() + mpa::kMaxPlanSeqs - 1) / mpa::kMaxPlanSeqs);
  return MPA_OK;
}

void mpa_default_rates(mpa_rates* r) {
  if (!r) return;
  // Least-squares fit (log error) to the phase times bench.py measured on
  // one MI355X for decode8b, lent, agentic, budget0/256/1024/4096 and
  // longctx (seed 0, each phase less the ~5 us of its event record); the
  // merge, few-key and wave figures are single kernel times from rocprofv3.
  // The append figures are fitted to the append phases alone: the
  // per-token launch from decode8b and budget0, the per-block launch (a
  // latency floor, then about 3.7 TB/s) from lent, budget4096 and longctx.
  r->append_fixed_us = 3.9;
  r->append_gbs = 545.0;
  r->append_block_us = 17.0;
  r->append_block_gbs = 3700.0;
  // decode: refitted to the decode half alone after its cache reads became
  // non-temporal (the fit puts the launch's fixed cost inside the rate)
  r->decode_fixed_us = 0.0;
  r->decode_gbs = 5880.0;
  r->decode_wave_gbs = 4.8;
  r->merge_us = 5.0;
  // prefill: refitted to the prefill half alone (lent, agentic, the budget
  // chunks, longctx) on two devices whose prefill rates differ by 5-7 %,
  // the mean of the two least-squares fits (12 + 1.80 per tile and 11.9 +
  // 1.76 against 12.1 + 1.85)
  r->prefill_wg_us = 12.0;
  r->prefill_tile_us = 1.80;
  r->prefill_merge_us = 3.0;
  r->prefill_merge_row_us = 1.6e-4;
  // A partitioned step's fixed cost beyond the model (the cross-stream waits,
  // and interference that the slowdown factor underrates on short steps):
  // fitted with coexec_slowdown, on a grid, to the four modes measured on
  // agentic, lent, budget4096, budget1024 and longctx, and on the TP4 shares
  // of agentic, lent and budget4096: the lowest mean regret of the
  // planner's choice with no choice slower than one stream is at slowdown
  // 1.10; the slowdown is one grid step above it (1.15), a margin for the
  // few percent that step times move between devices
  r->coexec_fixed_us = 130.0;
  // the few-key rows' second pass over their first key tile adds less than
  // a tile to one workgroup, which the makespan absorbs
  r->prefill_fixup_us = 0.0;
  r->prefill_slots = 256;
  // CU-partitioned co-execution (mpa_plan_coexec), measured on agentic, lent,
  // budget4096, budget1024 and longctx, each half alone on its CU set: the
  // decode half's speed on 1, 2 and 3 quarters of every XCD's CUs relative
  // to the whole device, the prefill half's likewise (faster than its share
  // of the CUs: fewer CUs contend for the same HBM and L2), medians over the
  // five; and the slowdown of the two halves side by side over the slower of
  // them alone (shared HBM, L2 and MALL)
  r->coexec_decode_q1 = 0.53;
  r->coexec_decode_q2 = 0.83;
  r->coexec_decode_q3 = 1.0;
  r->coexec_prefill_q1 = 0.33;
  r->coexec_prefill_q2 = 0.60;
  r->coexec_prefill_q3 = 0.73;
  r->coexec_slowdown = 1.15;
}

int mpa_predict_step(const mpa_shape* shape, const int32_t* seq_lens_host, const int32_t* qsl_host,
                     const mpa_rates* rates, mpa_step_time* out) {
  if (!out) return MPA_ERR_INVALID;
  mpa_rates def;
  mpa_default_rates(&def);
  const mpa_rates& r = rates ? *rates : def;
  Batch b;
  int rc = check_model_inputs(shape, seq_lens_host, qsl_host, r, &b);
  if (rc != MPA_OK) return rc;
  *out = model_step(shape, b, seq_lens_host, qsl_host, r);
  return MPA_OK;
}

int mpa_plan_coexec(const mpa_shape* shape, const int32_t* seq_lens_host, const int32_t* qsl_host,
                    const mpa_rates* rates, int32_t* mode, double* predicted_us) {
  if (!mode) return MPA_ERR_INVALID;
  mpa_rates def;
  mpa_default_rates(&def);
  const mpa_rates& r = rates ? *rates : def;
  Batch b;
  int rc = check_model_inputs(shape, seq_lens_host, qsl_host, r, &b);
  if (rc != MPA_OK) return rc;
  const double dfrac[4] = {1.0, r.coexec_decode_q1, r.coexec_decode_q2, r.coexec_decode_q3};
  const double pfrac[4] = {1.0, r.coexec_prefill_q3, r.coexec_prefill_q2, r.coexec_prefill_q1};
  if (!(r.coexec_slowdown >= 1.0)) return MPA_ERR_INVALID;
  for (int k = 1; k <= 3; ++k)
    if (!(dfrac[k] > 0) || !(pfrac[k] > 0)) return MPA_ERR_INVALID;
  if (!(r.coexec_fixed_us >= 0.0)) return MPA_ERR_INVALID;
  const mpa_step_time serial = model_step(shape, b, seq_lens_host, qsl_host, r);
  double t[4];
  t[0] = serial.decode_us + serial.prefill_us;
  // The prefill half on the (4 - k) / 4 of the CUs: its workgroups' makespan
  // on that share of the slots relative to all of them (more rounds when the
  // batch has few workgroups), times the per-CU speed measured on that share
  // (pfrac against the share itself), and never faster than alone on the
  // whole device.
  const std::vector<PrefillSplit> ps = prefill_splits(shape, b, seq_lens_host, qsl_host, 0);
  const double all_slots = prefill_time(shape, b, seq_lens_host, qsl_host, ps, r.prefill_wg_us, r.prefill_tile_us,
                                        r.prefill_slots, 0.0, 0.0);
  for (int k = 1; k <= 3; ++k) {
    if (b.decode.empty() || b.prefill.empty()) {
      t[k] = INFINITY;  // nothing to overlap
      continue;
    }
    const double share = (4 - k) / 4.0;
    const int slots = std::max(1, (int)lround(r.prefill_slots * share));
    const double rounds = prefill_time(shape, b, seq_lens_host, qsl_host, ps, r.prefill_wg_us, r.prefill_tile_us,
                                       slots, 0.0, 0.0) /
                          all_slots;
    const double prefill_k = serial.prefill_us * std::max(1.0, rounds * share / pfrac[k]);
    t[k] = std::max(serial.decode_us / dfrac[k], prefill_k) * r.coexec_slowdown + r.coexec_fixed_us;
  }
  int best = 0;
  for (int k = 1; k <= 3; ++k)
    if (t[k] < t[best]) best = k;
  *mode = best;
  if (predicted_us)
    for (int k = 0; k < 4; ++k) predicted_us[k] = t[k];
  return MPA_OK;
}

int mpa_partition_streams(int32_t mode, void** decode_stream, void** prefill_stream) {
  if (mode < 1 || mode > 3 || !decode_stream || !prefill_stream) return MPA_ERR_INVALID;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return MPA_ERR_HIP;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0 ||
      cus > 32 * kMaskWords)
    return MPA_ERR_HIP;
  static std::mutex lock;
  static hipStream_t made[64][3][2];
  std::lock_guard<std::mutex> guard(lock);
  hipStream_t* pair = made[dev][mode - 1];
  if (!pair[0]) {
    // CU i (the mask's numbering) goes to the decode half when (i / 8) % 4 <
    // mode: `mode` quarters of every XCD whether the numbering runs XCD by
    // XCD or interleaves them
    uint32_t dmask[kMaskWords] = {0}, pmask[kMaskWords] = {0};
    for (int i = 0; i < cus; ++i) ((i / 8) % 4 < mode ? dmask : pmask)[i / 32] |= 1u << (i % 32);
    const uint32_t words = (uint32_t)((cus + 31) / 32);
    hipStream_t d = nullptr, p = nullptr;
    if (hipExtStreamCreateWithCUMask(&d, words, dmask) != hipSuccess) return MPA_ERR_HIP;
    if (hipExtStreamCreateWithCUMask(&p, words, pmask) != hipSuccess) {
      (void)hipStreamDestroy(d);
      return MPA_ERR_HIP;
    }
    pair[0] = d;
    pair[1] = p;
  }
  *decode_stream = pair[0];
  *prefill_stream = pair[1];
  return MPA_OK;
}

size_t mpa_workspace_size(const mpa_shape* shape, const int32_t* seq_lens_host, const int32_t* qsl_host) {
  Batch b;
  if (check_batch(shape, seq_lens_host, qsl_host, nullptr, false, &b) != MPA_OK) return 0;
  const int split = choose_split(shape, b, seq_lens_host, qsl_host);
  bool any_split = false;
  for (int s : b.decode) any_split |= row_split(seq_lens_host[s], split).parts > 1;
  const long ditems = decode_items(shape, b, seq_lens_host, split);
  const long pitems = prefill_items(prefill_splits(shape, b, seq_lens_host, qsl_host, ditems), b, qsl_host);
  if (!any_split && pitems == 0) return 0;
  return workspace_bytes(shape, ditems + pitems);
}

int mpa_kv_append(const mpa_shape* shape, const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                  const int32_t* block_tables, const int32_t* seq_lens, const int32_t* query_start_loc,
                  const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                  const int32_t* block_tables_host, void* stream) {
  return run_append(shape, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host,
                    query_start_loc_host, block_tables_host, nullptr, stream);
}

int mpa_kv_append_rope(const mpa_shape* shape, void* q, const void* k_new, const void* v_new, void* k_cache,
                       void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                       const int32_t* query_start_loc, const int32_t* seq_lens_host,
                       const int32_t* query_start_loc_host, const int32_t* block_tables_host,
                       const float* rope_cos_sin, int32_t rope_dim, int32_t rope_max_pos, void* stream) {
  if (!shape) return MPA_ERR_INVALID;
  if (rope_dim <= 0 || rope_dim % 16 != 0 || rope_dim > shape->head_dim || rope_max_pos <= 0)
    return MPA_ERR_INVALID;
  if (shape->total_q_tokens > 0 && (!q || !rope_cos_sin)) return MPA_ERR_INVALID;
  if (seq_lens_host && shape->num_seqs > 0)
    for (int s = 0; s < shape->num_seqs; ++s)
      if (seq_lens_host[s] > rope_max_pos) return MPA_ERR_INVALID;  // a position past the table
  mpa::RopeArgs r;
  r.q = q;
  r.cos_sin = rope_cos_sin;
  r.hq = shape->num_q_heads;
  r.half = rope_dim / 2;
  return run_append(shape, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host,
                    query_start_loc_host, block_tables_host, &r, stream);
}

}  // extern "C"

namespace {

enum Phase { kDecode = 1, kPrefill = 2 };

int run_attention(int phases, const mpa_shape* shape, const void* q, const void* k_cache, const void* v_cache,
                  const int32_t* block_tables, const int32_t* seq_lens, const int32_t* query_start_loc,
                  const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                  const int32_t* block_tables_host, void* out, float* lse, void* workspace,
                  size_t workspace_bytes_given, void* stream, const void* k_new = nullptr,
                  const void* v_new = nullptr, bool validate_only = false) {
  Batch b;
  int rc = check_batch(shape, seq_lens_host, query_start_loc_host, block_tables_host, false, &b);
  if (rc != MPA_OK) return rc;
  if (!(phases & kDecode)) b.decode.clear();
  if (!(phases & kPrefill)) b.prefill.clear();
  if (b.decode.empty() && b.prefill.empty()) return MPA_OK;
  if (!q || !k_cache || !v_cache || !block_tables || !seq_lens || !query_start_loc || !out)
    return MPA_ERR_INVALID;
  // The split size depends on every decode row of the batch, whichever
  // phase runs, so that the phases together equal the mixed call exactly.
  // The workspace layout (decode partials, then prefill partials) is also
  // the whole batch's, so the two halves can run concurrently.
  Batch all;
  check_batch(shape, seq_lens_host, query_start_loc_host, nullptr, false, &all);
  const int split = choose_split(shape, all, seq_lens_host, query_start_loc_host);
  const long ditems = decode_items(shape, all, seq_lens_host, split);
  const std::vector<PrefillSplit> psplit =
      prefill_splits(shape, all, seq_lens_host, query_start_loc_host, ditems);
  const long items = ditems + prefill_items(psplit, all, query_start_loc_host);
  bool any_split = false;
  for (int s : b.decode) any_split |= row_split(seq_lens_host[s], split).parts > 1;
  if (!b.prefill.empty())
    for (const auto& ps : psplit) any_split |= ps.nsplit > 1;
  if (any_split) {
    const size_t need = workspace_bytes(shape, items);
    if (!workspace || workspace_bytes_given < need || ((uintptr_t)workspace & 15) != 0) return MPA_ERR_WORKSPACE;
  }
  mpa::AttnArgs a;
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.block_tables = block_tables;
  a.seq_lens = seq_lens;
  a.qsl = query_start_loc;
  a.out = out;
  a.lse = lse;
  a.ws_o = any_split ? static_cast<float*>(workspace) : nullptr;
  a.ws_ml = any_split ? a.ws_o + (size_t)items * shape->num_q_heads * shape->head_dim : nullptr;
  a.hq = shape->num_q_heads;
  a.hkv = shape->num_kv_heads;
  a.mb = shape->max_blocks_per_seq;
  a.nb = shape->num_blocks;
  // fp8 caches: the key scale folds into the softmax scale, the value scale
  // into the output (and the split partials)
  const bool fp8 = shape->dtype == MPA_FP8;
  a.scale_log2 = shape->scale * 1.4426950408889634f * (fp8 ? shape->k_scale : 1.f);
  a.v_scale = fp8 ? shape->v_scale : 1.f;
  a.k_new = k_new;
  a.v_new = v_new;
  a.inv_k_scale = fp8 ? 1.f / shape->k_scale : 1.f;
  a.inv_v_scale = fp8 ? 1.f / shape->v_scale : 1.f;
  if (validate_only) return MPA_OK;
  hipStream_t st = (hipStream_t)stream;
  clear_stale_hip_error();

  // Decode rows, in launches of up to kMaxPlanSeqs sequences.
  std::vector<mpa::DecodePlan> dplans;
  {
    long base = 0;
    for (size_t c0 = 0; c0 < b.decode.size(); c0 += mpa::kMaxPlanSeqs) {
      mpa::DecodePlan p;
      memset(&p, 0, sizeof(p));
      const size_t c1 = std::min(b.decode.size(), c0 + mpa::kMaxPlanSeqs);
      p.n_seqs = (int32_t)(c1 - c0);
      p.item_base = (int32_t)base;
      int acc = 0;
      for (size_t k = c0; k < c1; ++k) {
        const int s = b.decode[k];
        const RowSplit rs = row_split(seq_lens_host[s], split);
        p.seq[k - c0] = s;
        p.split_tokens[k - c0] = rs.tokens;
        p.item_start[k - c0] = acc;
        acc += rs.parts;
      }
      p.item_start[c1 - c0] = acc;
      base += acc;
      dplans.push_back(p);
    }
  }
  for (const auto& p : dplans) {
    hipError_t e = mpa::launch_decode(a, p, p.item_start[p.n_seqs], shape->dtype, shape->head_dim, st);
    if (e != hipSuccess) return MPA_ERR_HIP;
  }
  if (any_split) {
    for (const auto& p : dplans) {
      hipError_t e = mpa::launch_merge(a, p, shape->dtype, shape->head_dim, st);
      if (e != hipSuccess) return MPA_ERR_HIP;
    }
  }
  // Prefill chunks (b.prefill is all.prefill or empty), in launches of up to
  // kMaxPrefillSeqs; KV-split chunks are merged after their launch.
  const int qt = q_tile(shape);
  for (size_t c0 = 0; c0 < b.prefill.size(); c0 += mpa::kMaxPrefillSeqs) {
    mpa::PrefillPlan p;
    memset(&p, 0, sizeof(p));
    const size_t c1 = std::min(b.prefill.size(), c0 + mpa::kMaxPrefillSeqs);
    p.n_seqs = (int32_t)(c1 - c0);
    p.q_tile = qt;
    int acc = 0, rows = 0;
    for (size_t k = c0; k < c1; ++k) {
      const int s = b.prefill[k];
      const int C = query_start_loc_host[s + 1] - query_start_loc_host[s];
      const PrefillSplit& ps = psplit[k];
      p.seq[k - c0] = s;
      p.tile_start[k - c0] = acc;
      p.nsplit[k - c0] = ps.nsplit;
      p.split_tiles[k - c0] = ps.tiles;
      p.item_base[k - c0] = (int32_t)ps.item_base;
      p.row_start[k - c0] = rows;
      acc += (C + qt - 1) / qt * ps.nsplit;
      if (ps.nsplit > 1) rows += C;
    }
    p.tile_start[c1 - c0] = acc;
    p.row_start[c1 - c0] = rows;
    hipError_t e = mpa::launch_prefill(a, p, acc, shape->dtype, shape->head_dim, st);
    if (e != hipSuccess) return MPA_ERR_HIP;
    if (rows > 0) {
      e = mpa::launch_prefill_merge(a, p, shape->dtype, shape->head_dim, st);
      if (e != hipSuccess) return MPA_ERR_HIP;
    }
  }
  return MPA_OK;
}

// The append and the attention of the rows in `phases`, in one call: the
// attention's checks (the workspace included) and the append's run first,
// so an error means nothing was launched; then the multi-token rows' block
// append (prefill phase), and the attention, whose decode kernel writes the
// decode rows' new tokens itself.
int run_fused(int phases, const mpa_shape* shape, const void* q, const void* k_new, const void* v_new,
              void* k_cache, void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
              const int32_t* query_start_loc, const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
              const int32_t* block_tables_host, void* out, float* lse, void* workspace, size_t workspace_bytes_given,
              void* stream) {
  int rc = run_attention(phases, shape, q, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host,
                         query_start_loc_host, block_tables_host, out, lse, workspace, workspace_bytes_given, stream,
                         nullptr, nullptr, true);
  if (rc != MPA_OK) return rc;
  if (shape->total_q_tokens > 0 && (!k_new || !v_new)) return MPA_ERR_INVALID;
  if (phases & kPrefill) {
    rc = run_append(shape, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host,
                    query_start_loc_host, block_tables_host, nullptr, stream, true);
    if (rc != MPA_OK) return rc;
  } else if (debug_checks()) {
    rc = check_append_slots(shape, seq_lens_host, query_start_loc_host, block_tables_host);
    if (rc != MPA_OK) return rc;
  }
  return run_attention(phases, shape, q, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host,
                       query_start_loc_host, block_tables_host, out, lse, workspace, workspace_bytes_given, stream,
                       k_new, v_new);
}

}  // namespace

extern "C" {

int mpa_mixed_paged_attention(const mpa_shape* shape, const void* q, const void* k_cache, const void* v_cache,
                              const int32_t* block_tables, const int32_t* seq_lens, const int32_t* query_start_loc,
                              const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                              const int32_t* block_tables_host, void* out, float* lse, void* workspace,
                              size_t workspace_bytes_given, void* stream) {
  return run_attention(kDecode | kPrefill, shape, q, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
                       seq_lens_host, query_start_loc_host, block_tables_host, out, lse, workspace,
                       workspace_bytes_given, stream);
}

int mpa_append_attention(const mpa_shape* shape, const void* q, const void* k_new, const void* v_new,
                         void* k_cache, void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                         const int32_t* query_start_loc, const int32_t* seq_lens_host,
                         const int32_t* query_start_loc_host, const int32_t* block_tables_host, void* out,
                         float* lse, void* workspace, size_t workspace_bytes_given, void* stream) {
  return run_fused(kDecode | kPrefill, shape, q, k_new, v_new, k_cache, v_cache, block_tables, seq_lens,
                   query_start_loc, seq_lens_host, query_start_loc_host, block_tables_host, out, lse, workspace,
                   workspace_bytes_given, stream);
}

int mpa_append_decode_attention(const mpa_shape* shape, const void* q, const void* k_new, const void* v_new,
                                void* k_cache, void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                                const int32_t* query_start_loc, const int32_t* seq_lens_host,
                                const int32_t* query_start_loc_host, const int32_t* block_tables_host, void* out,
                                float* lse, void* workspace, size_t workspace_bytes_given, void* stream) {
  return run_fused(kDecode, shape, q, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
                   seq_lens_host, query_start_loc_host, block_tables_host, out, lse, workspace,
                   workspace_bytes_given, stream);
}

int mpa_append_prefill_attention(const mpa_shape* shape, const void* q, const void* k_new, const void* v_new,
                                 void* k_cache, void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                                 const int32_t* query_start_loc, const int32_t* seq_lens_host,
                                 const int32_t* query_start_loc_host, const int32_t* block_tables_host, void* out,
                                 float* lse, void* workspace, size_t workspace_bytes_given, void* stream) {
  return run_fused(kPrefill, shape, q, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
                   seq_lens_host, query_start_loc_host, block_tables_host, out, lse, workspace,
                   workspace_bytes_given, stream);
}

int mpa_decode_attention(const mpa_shape* shape, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* block_tables, const int32_t* seq_lens, const int32_t* query_start_loc,
                         const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                         const int32_t* block_tables_host, void* out, float* lse, void* workspace,
                         size_t workspace_bytes_given, void* stream) {
  return run_attention(kDecode, shape, q, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
                       seq_lens_host, query_start_loc_host, block_tables_host, out, lse, workspace,
                       workspace_bytes_given, stream);
}

int mpa_prefill_attention(const mpa_shape* shape, const void* q, const void* k_cache, const void* v_cache,
                          const int32_t* block_tables, const int32_t* seq_lens, const int32_t* query_start_loc,
                          const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                          const int32_t* block_tables_host, void* out, float* lse, void* workspace,
                          size_t workspace_bytes_given, void* stream) {
  return run_attention(kPrefill, shape, q, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
                       seq_lens_host, query_start_loc_host, block_tables_host, out, lse, workspace,
                       workspace_bytes_given, stream);
}

}  // extern "C"
