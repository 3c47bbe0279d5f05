/*
 * mpa.h -- mixed prefill+decode paged attention for one MI355X (gfx950).
 *
 * One serving iteration of a decode node that lends compute to prefill work
 * (Crossflow, arxiv 2609.27085): the decode node takes a whole request,
 * reuses its resident prefix and runs the remaining prompt tokens as chunks
 * inside the same batch as its running decode rows (section 4.4, "Spilled-
 * request execution"; section 5, the local prefill queue and the mixed
 * prefill/decode batch).  This library is that iteration's attention step:
 * append the step's new K/V to a paged cache, then attend for every query
 * row of the varlen batch through per-sequence block tables.
 *
 * ---------------------------------------------------------------------------
 * Batch description (all int32):
 *   S                  number of sequences in the step
 *   query_start_loc    [S+1], query_start_loc[0] = 0, non-decreasing,
 *                      query_start_loc[S] = T (total query tokens).  Sequence
 *                      s owns query rows query_start_loc[s] .. [s+1]-1.
 *   seq_lens           [S], KV length of sequence s AFTER this step's append.
 *                      q_len(s) = query_start_loc[s+1] - query_start_loc[s]
 *                      must satisfy 0 <= q_len(s) <= seq_lens[s].
 *   block_tables       [S][max_blocks_per_seq], row-major; entry j of row s is
 *                      the physical block holding logical positions
 *                      16*j .. 16*j+15 of sequence s.  Only the first
 *                      ceil(seq_lens[s] / 16) entries of a row are read.
 *
 * Positions and the causal rule: sequence s has a cached prefix of
 * P = seq_lens[s] - q_len(s) tokens; its new token i (query row
 * query_start_loc[s] + i) sits at logical position P + i and attends keys
 * 0 .. P + i inclusive.  q_len = 1 is a decode row (it sees the whole
 * context); q_len > 1 is a prefill chunk on the cached prefix; q_len = 0
 * sequences are skipped.  Query head h reads KV head h / (Hq / Hkv).
 *
 * Tensors (device memory, dense, row-major; element type = shape.dtype):
 *   q        [T][Hq][d]
 *   k_new    [T][Hkv][d]      the step's new keys, row t = query row t
 *   v_new    [T][Hkv][d]
 *   out      [T][Hq][d]
 *   lse      [T][Hq] float32, natural log of each row's softmax denominator
 *   k_cache  [num_blocks][Hkv][d/X][16][X]   X = 8 (bf16, fp8) or 4 (f32)
 *   v_cache  [num_blocks][Hkv][d][16]
 * i.e. key element (block b, head h, slot t, dim i) is at
 * k_cache[b][h][i/X][t][i%X] and value element (b, h, t, i) at
 * v_cache[b][h][i][t].  A (block, head) is one contiguous 16*d-element
 * granule of each cache.  Shared (prefix) blocks may appear in several
 * rows; the slots a step appends to must be distinct.
 *
 * Supported: dtype bf16 or f32 (the caches, q, k_new, v_new and out all in
 * that type), or fp8 (the caches hold OCP FP8 E4M3 codes, one byte per
 * element, with one scale per cache; q, k_new, v_new and out are bf16);
 * head_dim 64 or 128, block_size 16, Hq a multiple of Hkv with
 * Hq / Hkv <= 16.
 *
 * fp8 caches: the paper is silent on cache precision.  A key value x is
 * stored as the E4M3 code nearest to x * (1 / k_scale) -- the reciprocal
 * and the product each rounded to float32 -- with ties to the even
 * mantissa and magnitudes past 448 saturated to 448 (NaN stays NaN); it is
 * read back as code value * k_scale (values likewise with v_scale).  E4M3:
 * sign bit, 4-bit exponent with bias 7, 3-bit mantissa, subnormals m*2^-9,
 * S.1111.111 = NaN, no infinity.
 *
 * Conventions:
 *  - The caller owns every buffer.  The library allocates nothing and keeps
 *    no state between calls; calls on different streams are independent.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream).  The host arrays are read before the call returns.
 *  - Every check runs before the first launch: an error return means that
 *    nothing was launched and no device memory was touched.  Devices ids in
 *    block_tables that the host did not check (block_tables_host == NULL)
 *    are also guarded on the device: a block id outside [0, num_blocks)
 *    is never dereferenced; the rows that needed it come out as NaN, and
 *    the append skips the token.
 *  - Cache slots at positions >= seq_lens[s] and blocks no row references
 *    never influence any output, whatever they hold (NaN and Inf included).
 * ---------------------------------------------------------------------------
 */
#ifndef MPA_H_
#define MPA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MPA_OK = 0,
  MPA_ERR_INVALID = -1,     /* malformed arguments or batch metadata */
  MPA_ERR_UNSUPPORTED = -2, /* a shape or dtype this build does not handle */
  MPA_ERR_WORKSPACE = -3,   /* workspace missing, smaller than required or misaligned */
  MPA_ERR_HIP = -4,         /* a HIP launch reported an error */
  MPA_ERR_SCRATCH = -5      /* mpa_append_attention_noalloc: the batch needs more than MPA_SCRATCH_BYTES */
} mpa_status;

/* Size of the library's fixed device array behind mpa_append_attention_noalloc. */
#define MPA_SCRATCH_BYTES ((size_t)256 << 20)

typedef enum { MPA_BF16 = 0, MPA_F32 = 1, MPA_FP8 = 2 } mpa_dtype;

typedef struct {
  int32_t num_seqs;           /* S */
  int32_t num_q_heads;        /* Hq */
  int32_t num_kv_heads;       /* Hkv */
  int32_t head_dim;           /* d: 64 or 128 */
  int32_t block_size;         /* must be 16 */
  int32_t num_blocks;         /* physical blocks in each cache */
  int32_t max_blocks_per_seq; /* row stride of block_tables */
  int32_t total_q_tokens;     /* T = query_start_loc[S] */
  float scale;                /* softmax scale, finite and > 0, e.g. 1/sqrt(d) */
  int32_t dtype;              /* mpa_dtype */
  float k_scale;              /* fp8: key cache scale, finite and > 0 (else unused) */
  float v_scale;              /* fp8: value cache scale, finite and > 0 (else unused) */
} mpa_shape;

/*
 * Append the step's new keys and values to the paged cache.
 *
 * Defines: new token i of sequence s (query row query_start_loc[s] + i) is
 * position p = seq_lens[s] - q_len(s) + i, and its Hkv*d key and value
 * elements are copied, bit for bit, to slot p % 16 of block
 * block_tables[s][p / 16] (paper, section 4.4: the chunk's KV is
 * materialised on top of the reused prefix; section 2.1: decode extends the
 * KV cache by one token per step).  No other cache element changes.
 *
 * k_new, v_new      device [T][Hkv][d]
 * k_cache, v_cache  device caches (layout above), written in place
 * block_tables, seq_lens, query_start_loc        device copies
 * seq_lens_host, query_start_loc_host            host copies (must match)
 * block_tables_host host copy [S][max_blocks_per_seq] or NULL; when given,
 *                   every block id the step uses is checked on the host.
 * With MPA_DEBUG=1 in the environment (read at each call) the host also
 * checks that the slots written are pairwise distinct and that none holds a
 * key a sequence of the step reads (prefix blocks shared between sequences
 * are read-only); this needs block_tables_host and visits every key of the
 * step.  A violation, or a missing block_tables_host, gives MPA_ERR_INVALID.
 * Returns MPA_OK, or an error code with nothing launched.
 */
int mpa_kv_append(const mpa_shape* shape, const void* k_new, const void* v_new, void* k_cache,
                  void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                  const int32_t* query_start_loc, const int32_t* seq_lens_host,
                  const int32_t* query_start_loc_host, const int32_t* block_tables_host,
                  void* stream);

/*
 * mpa_kv_append with the rotary position embedding applied on the way:
 * every new token's query row (all Hq heads, in place) and key row are
 * rotated by the token's position p = seq_lens[s] - q_len(s) + i before the
 * key is written to the cache; values are appended unchanged.  The paper
 * describes neither its models' position encoding nor such a kernel; this
 * is the standard rotary embedding in the rotate-half form, fused into the
 * step that writes the cache.  With R = rope_dim and, for j < R/2,
 * (c, s) = rope_cos_sin[p][j]:
 *   y[j]       = x[j] * c - x[j + R/2] * s
 *   y[j + R/2] = x[j + R/2] * c + x[j] * s
 * and y[i] = x[i] for i >= R (partial rotary when R < d).  Each product and
 * each sum is rounded to float32 (no fused multiply-add), the result to the
 * row's element type (bf16: nearest even).  With an fp8 cache the rotated
 * key, so rounded to bf16, is then stored as a plain new key would be (the
 * E4M3 code of y * (1 / k_scale)); q stays bf16.
 *
 * q                 device [T][Hq][d], rotated in place
 * rope_cos_sin      device float32 [rope_max_pos][R/2][2] (cos, sin), e.g.
 *                   cos/sin of p * base^(-2j/R); any table (scaled variants
 *                   included) may be passed
 * rope_dim          R: a multiple of 16, at most head_dim
 * rope_max_pos      rows of the table; every position must be below it
 *                   (checked against seq_lens_host)
 * Other arguments, ownership and errors as for mpa_kv_append.
 */
int mpa_kv_append_rope(const mpa_shape* shape, void* q, const void* k_new, const void* v_new, void* k_cache,
                       void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                       const int32_t* query_start_loc, const int32_t* seq_lens_host,
                       const int32_t* query_start_loc_host, const int32_t* block_tables_host,
                       const float* rope_cos_sin, int32_t rope_dim, int32_t rope_max_pos, void* stream);

/*
 * Bytes of device workspace that mpa_mixed_paged_attention needs for this
 * batch: the split-K partial results of long decode rows, and of prefill
 * chunks whose cached prefix is split across workgroups (short bf16 chunks
 * on long prefixes, when the batch's prefill tiles alone would leave most of
 * the device idle).  Depends only on the shape and the host metadata.
 * Returns 0 for an invalid batch, and when nothing is split.
 */
size_t mpa_workspace_size(const mpa_shape* shape, const int32_t* seq_lens_host,
                          const int32_t* query_start_loc_host);

/*
 * Attention for every query row of the mixed batch, reading K/V only from
 * the (already appended) cache.
 *
 * Defines: for query row t of sequence s at position p and query head h,
 *   out[t][h] = sum_{j<=p} softmax_j(scale * q[t][h] . k_j) v_j
 * over sequence s's keys k_j, v_j (KV head h / (Hq/Hkv)), and
 *   lse[t][h] = log sum_{j<=p} exp(scale * q[t][h] . k_j).
 * The paper (section 2.1) has decode re-read the growing KV cache each
 * step and (section 4.4, section 5) batches prefill chunks on cached
 * prefixes with those decode rows; it does not write the formula out --
 * this is standard scaled dot-product attention under the causal rule above.
 *
 * Decode rows (q_len = 1) run as split-K over KV blocks with an LSE merge;
 * prefill chunks (q_len > 1) run as causal MFMA tiles, their cached prefix
 * also split (and merged the same way) when the chunks are short.
 *
 * q                 device [T][Hq][d]
 * out               device [T][Hq][d], written for every row of every
 *                   sequence with q_len > 0
 * lse               device [T][Hq] float32, or NULL
 * workspace         device scratch of at least mpa_workspace_size() bytes,
 *                   16-byte aligned
 *                   (may be NULL when that is 0); contents on entry unused
 * Other arguments as for mpa_kv_append.
 */
int mpa_mixed_paged_attention(const mpa_shape* shape, const void* q, const void* k_cache,
                              const void* v_cache, const int32_t* block_tables,
                              const int32_t* seq_lens, const int32_t* query_start_loc,
                              const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                              const int32_t* block_tables_host, void* out, float* lse,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * One whole step of the mixed iteration in one call: mpa_kv_append followed
 * by mpa_mixed_paged_attention on the same batch, with results (cache
 * contents, out, lse) bit-identical to the two calls.  The decode rows
 * extend the KV cache by one token each (section 2.1) and the chunk's KV is
 * materialised on the reused prefix before it is attended to (section 4.4);
 * here a decode row's new token is written by the decode kernel itself --
 * by the wave that reads the row's last split, the only one whose keys
 * include it -- which saves the per-token append launch, while multi-token
 * rows keep their own append launch ahead of the prefill kernel.
 *
 * k_new, v_new      device [T][Hkv][d] (bf16 for fp8 caches), as for
 *                   mpa_kv_append; may be NULL only when T == 0
 * k_cache, v_cache  written (the new tokens) and read
 * Other arguments as for mpa_mixed_paged_attention.  Every check of both
 * calls (the workspace included) runs before the first launch: an error
 * return means nothing was launched.  With MPA_DEBUG=1 the append's slot
 * checks apply.
 */
int mpa_append_attention(const mpa_shape* shape, const void* q, const void* k_new, const void* v_new,
                         void* k_cache, void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                         const int32_t* query_start_loc, const int32_t* seq_lens_host,
                         const int32_t* query_start_loc_host, const int32_t* block_tables_host, void* out,
                         float* lse, void* workspace, size_t workspace_bytes, void* stream);

/*
 * mpa_append_attention without a workspace argument, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  The step's split-K
 * partial results live in a fixed device array inside the library,
 * MPA_SCRATCH_BYTES (256 MiB) on each device the library runs on, held
 * until the process ends; its device address is looked up (with
 * hipGetSymbolAddress) on the first call on each device.  The call itself
 * allocates no device memory.
 *
 * Arguments, results (bit-identical to mpa_append_attention) and checks as
 * for mpa_append_attention.  A batch for which mpa_workspace_size exceeds
 * MPA_SCRATCH_BYTES returns MPA_ERR_SCRATCH with nothing launched; use
 * mpa_append_attention with a workspace for it.  Every call on a device
 * shares that device's array: calls that overlap on one device (two
 * streams, two threads) race on it and must be serialised by the caller.
 * No part of the array needs to start at zero.
 */
int mpa_append_attention_noalloc(const mpa_shape* shape, const void* q, const void* k_new, const void* v_new,
                                 void* k_cache, void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                                 const int32_t* query_start_loc, const int32_t* seq_lens_host,
                                 const int32_t* query_start_loc_host, const int32_t* block_tables_host, void* out,
                                 float* lse, void* stream);

/*
 * The two halves of mpa_append_attention, as mpa_decode_attention and
 * mpa_prefill_attention are of mpa_mixed_paged_attention: the decode half
 * appends and attends the rows of sequences with q_len == 1 (the decode
 * kernel writing their new tokens), the prefill half appends the new tokens
 * of sequences with q_len > 1 (by cache block) and then attends their rows.
 * Same arguments and checks as mpa_append_attention; running both gives its
 * results bit for bit.  The halves write disjoint cache slots, rows and
 * workspace, read none of each other's new keys, and may run concurrently.
 */
int mpa_append_decode_attention(const mpa_shape* shape, const void* q, const void* k_new, const void* v_new,
                                void* k_cache, void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                                const int32_t* query_start_loc, const int32_t* seq_lens_host,
                                const int32_t* query_start_loc_host, const int32_t* block_tables_host, void* out,
                                float* lse, void* workspace, size_t workspace_bytes, void* stream);
int mpa_append_prefill_attention(const mpa_shape* shape, const void* q, const void* k_new, const void* v_new,
                                 void* k_cache, void* v_cache, const int32_t* block_tables, const int32_t* seq_lens,
                                 const int32_t* query_start_loc, const int32_t* seq_lens_host,
                                 const int32_t* query_start_loc_host, const int32_t* block_tables_host, void* out,
                                 float* lse, void* workspace, size_t workspace_bytes, void* stream);

/*
 * The two halves of mpa_mixed_paged_attention, for callers that time them
 * separately or run them on two streams: mpa_decode_attention computes only
 * the rows of sequences with q_len == 1, mpa_prefill_attention only the rows
 * of sequences with q_len > 1.  Arguments and contracts are those of
 * mpa_mixed_paged_attention (the workspace is sized for the whole batch by
 * mpa_workspace_size; each half uses its own disjoint part of it); both
 * halves read the whole batch's metadata, so running both gives results
 * bit-identical to the mixed call.  The two write disjoint rows of out and
 * lse and disjoint workspace, and may run concurrently.
 */
int mpa_decode_attention(const mpa_shape* shape, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* block_tables, const int32_t* seq_lens, const int32_t* query_start_loc,
                         const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                         const int32_t* block_tables_host, void* out, float* lse, void* workspace,
                         size_t workspace_bytes, void* stream);

int mpa_prefill_attention(const mpa_shape* shape, const void* q, const void* k_cache, const void* v_cache,
                          const int32_t* block_tables, const int32_t* seq_lens, const int32_t* query_start_loc,
                          const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                          const int32_t* block_tables_host, void* out, float* lse, void* workspace,
                          size_t workspace_bytes, void* stream);

/* Static description of a status code. */
const char* mpa_status_string(int status);

/*
 * Plan statistics for a batch (host only; launches nothing): how the
 * library splits decode rows and tiles prefill chunks.
 */
typedef struct {
  int32_t num_decode_seqs;   /* sequences with q_len == 1 */
  int32_t num_prefill_seqs;  /* sequences with q_len > 1 */
  int32_t split_tokens;      /* nominal KV tokens per decode split: a row of L keys is cut into
                                ceil(L / split_tokens) parts of equal size, rounded up to whole
                                blocks (the last part ends at L) */
  int32_t num_decode_items;  /* (sequence, split) work items */
  int32_t num_prefill_tiles; /* (sequence, query tile, KV split, KV head) work items */
  int32_t decode_launches;   /* decode kernel launches (sequence chunks) */
  int32_t prefill_max_splits; /* most KV splits of any prefill chunk (0: no chunk) */
} mpa_plan_info;

int mpa_get_plan_info(const mpa_shape* shape, const int32_t* seq_lens_host,
                      const int32_t* query_start_loc_host, mpa_plan_info* info);

/*
 * Step-time model (host only; launches nothing).
 *
 * The paper has a decode node lend compute to spilled prefill under a lease
 * whose compute credit is counted in units the backend can bound, such as
 * token chunks (section 4.2), and admits a spill only when its predicted
 * service time under that lease beats the default path (section 4.3); it
 * stresses that the spare capacity beside a decode batch is nonlinear in the
 * batch's shape (section 3.2).  mpa_predict_step gives that service time for
 * this library: the device time of one step -- mpa_kv_append then
 * mpa_mixed_paged_attention on one stream -- predicted from the library's
 * own plan for the batch (decode splits, prefill query tiles, KV splits,
 * launches) and a few measured rates:
 *
 *   append  = per launch for single-token sequences: append_fixed_us +
 *             (bytes read and written) / append_gbs; per launch for
 *             multi-token sequences: max(append_block_us, bytes /
 *             append_block_gbs)
 *   decode  = per launch: decode_fixed_us + max(KV bytes / decode_gbs,
 *             largest wave's KV bytes / decode_wave_gbs), plus merge_us per
 *             launch when a row is split
 *   prefill = per launch: the makespan of its workgroups, each taking
 *             prefill_wg_us + prefill_tile_us per 64-key tile, dealt in
 *             launch order to prefill_slots workgroup slots; plus, per
 *             launch with a KV-split chunk, prefill_merge_us +
 *             prefill_merge_row_us per partial (token, q head, split) row;
 *             plus prefill_fixup_us when a chunk sits on a prefix shorter
 *             than 64 tokens (its first key tile is passed twice for the
 *             rows that see at most 64 keys; 0 in the default rates)
 *
 * Rates are in microseconds and GB/s (1e9 bytes/s).  mpa_default_rates
 * fills in figures measured on one MI355X with bench.py.  Only bf16 caches
 * are modelled: MPA_ERR_UNSUPPORTED for f32 and fp8.
 */
typedef struct {
  double append_fixed_us;
  double append_gbs;
  double decode_fixed_us;
  double decode_gbs;
  double decode_wave_gbs;
  double merge_us;
  double prefill_wg_us;
  double prefill_tile_us;
  double prefill_merge_us;
  double prefill_fixup_us;
  int32_t prefill_slots;
  double append_block_us;
  double append_block_gbs;
  double coexec_decode_q1;   /* decode half's speed on 1/4 of every XCD's CUs, relative to all */
  double coexec_decode_q2;   /* ... on 1/2 */
  double coexec_decode_q3;   /* ... on 3/4 */
  double coexec_prefill_q1;  /* prefill half's speed on 1/4 of every XCD's CUs, relative to all */
  double coexec_prefill_q2;  /* ... on 1/2 */
  double coexec_prefill_q3;  /* ... on 3/4 */
  double coexec_slowdown;    /* two halves side by side over the slower one alone (>= 1) */
  double prefill_merge_row_us; /* KV-split merge, per partial (token, q head, split) row */
  double coexec_fixed_us;      /* fixed cost of a step run on partitioned streams (>= 0) */
} mpa_rates;

typedef struct {
  double append_us;
  double decode_us;
  double prefill_us;
  double step_us; /* their sum: the three phases run one after the other */
} mpa_step_time;

void mpa_default_rates(mpa_rates* rates);

/* rates may be NULL (the defaults).  Returns MPA_OK or an error code with
 * *out untouched. */
int mpa_predict_step(const mpa_shape* shape, const int32_t* seq_lens_host,
                     const int32_t* query_start_loc_host, const mpa_rates* rates,
                     mpa_step_time* out);

/*
 * How to run the step's two attention halves (mpa_decode_attention and
 * mpa_prefill_attention), chosen per step.  The paper runs spilled prefill
 * beside decode either as a chunked mixed batch or, in its PDMUX executor,
 * on a spatial partition of the GPU; both are backends of one executor
 * interface (section 5).  Here mode 0 runs the halves one after the other
 * on one stream (as mpa_mixed_paged_attention does); mode k = 1, 2, 3 runs
 * them concurrently, the decode half on k quarters of every XCD's CUs and
 * the prefill half on the rest (mpa_partition_streams).  The outputs are
 * bit-identical in every mode.  The predicted attention time of mode k is
 *   mode 0: decode + prefill of mpa_predict_step
 *   mode k: max(decode / coexec_decode_qk, prefill_k) * coexec_slowdown
 *           + coexec_fixed_us
 * with prefill_k = prefill * max(1, rounds_k * s / coexec_prefill_q(4-k)),
 * s = (4 - k) / 4 the prefill half's share of the CUs and rounds_k the
 * makespan of the prefill workgroups on s * prefill_slots slots over that on
 * all of them (infinite when the step lacks decode rows or prefill chunks).
 *
 * mode          out: the mode with the shortest predicted time
 * predicted_us  out, may be NULL: double[4], the prediction per mode
 * Errors as for mpa_predict_step (bf16 caches only).
 */
int mpa_plan_coexec(const mpa_shape* shape, const int32_t* seq_lens_host, const int32_t* query_start_loc_host,
                    const mpa_rates* rates, int32_t* mode, double* predicted_us);

/*
 * The two streams of partition mode 1..3 on the current device: the decode
 * half's, restricted to `mode` quarters of every XCD's CUs, and the prefill
 * half's, restricted to the other CUs.  Created at the first request (per
 * device and mode, default priority) and kept until the process ends; the
 * caller orders them against its own stream (events) and never destroys
 * them.  Returns MPA_ERR_INVALID for another mode, MPA_ERR_HIP when the
 * runtime refuses.
 */
int mpa_partition_streams(int32_t mode, void** decode_stream, void** prefill_stream);

/*
 * Measurement probes (not part of the attention path).  They measure the
 * device's sustained rate on the two resources the step is bound by:
 * decode rows on HBM reads, prefill chunks on dense bf16 matrix-core work
 * (the paper's split of decode as memory bound and prefill as compute
 * bound, section 2.1), so that a kernel's rate can also be stated against a
 * measured peak.  Both launch one kernel on `stream`, allocate nothing, and
 * return MPA_OK, MPA_ERR_INVALID (nothing launched) or MPA_ERR_HIP.
 *
 * mpa_probe_stream_read: reads every byte of buf once with 16-byte non-temporal loads.
 *   buf    device, 16-byte aligned, `bytes` long (a multiple of 16, > 0)
 *   sink   device uint32_t[1]; written only when the data's XOR hits one
 *          fixed value (it keeps the loads), so its contents are unspecified
 *
 * mpa_probe_mfma_bf16: 1,024 workgroups of four waves (four per SIMD), each
 *   wave running `iters` rounds of four independent 32x32x16 bf16 MFMAs.
 *   sink   device float[1], never written in practice
 *   flops  host out, may be NULL: the launch's multiply-add work, 2 flops each
 */
int mpa_probe_stream_read(const void* buf, size_t bytes, uint32_t* sink, void* stream);
int mpa_probe_mfma_bf16(int32_t iters, float* sink, double* flops, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MPA_H_ */
