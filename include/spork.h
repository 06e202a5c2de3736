/*
 * spork.h -- C ABI of libspork: the forked-decode hot path of SPORK
 * (Self-Speculative Forking, arXiv 2607.03333) on AMD MI355X (gfx950).
 *
 * What the library computes
 *   - spork_fork: a probe thread forked from a main thread reuses the main
 *     thread's prefix KV blocks in place (design D1, Section 4.1: the probe's
 *     prefill becomes a prefix-cache hit). Blocks are shared through a
 *     reference-counted block table and copied on first write.
 *   - spork_attn_decode: one decode step of attention for a batch of main and
 *     probe threads over their paged KV. Threads of one fork group share their
 *     common prefix; its KV is streamed once per group, each thread's private
 *     suffix once per thread, and the parts are merged by log-sum-exp.
 *   - spork_verify_accept: the D3 step (Section 4.3): the rejected probe's
 *     tokens enter the main thread as K draft rows with a causal rule over the
 *     drafts; the greedy token of every verify row is the lowest index of its
 *     row maximum, and the accepted length is the longest draft prefix that
 *     equals the greedy tokens (decoding resumes after the first mismatch).
 *   - spork_probe_confidence: design D2's gate (Section 4.2): the top-1
 *     log-probability of every probe position and, per probe, the smallest
 *     top-1 probability over its tool-name span without the span's first
 *     token, compared with a threshold.
 *   - spork_ngram_propose: the n-gram (prompt-lookup) draft proposer of the
 *     engine's n-gram speculative decoding (Sections 4.3 and 6.1), a second
 *     source of the drafts spork_verify_accept checks.
 *
 * Conventions
 *   - Every entry point returns SPORK_OK (0) or a negative status and never
 *     throws or aborts; spork_last_error() gives a message for the calling
 *     thread's last failure.
 *   - Arguments are validated before anything is launched or changed: on an
 *     error no kernel is launched and the block manager is unchanged.
 *   - "host" pointers are CPU memory; "device" pointers are GPU memory of the
 *     current HIP device. All device memory is owned by the caller; launches go
 *     on the caller's stream and the library never synchronises it. Results
 *     are valid once that stream has been synchronised.
 *   - Objects (spork_cache, spork_plan) are not thread-safe; callers serialise
 *     calls on one object.
 *
 * KV pool layout (both pools have num_blocks blocks of block_size tokens):
 *   K pool: [num_blocks][Hkv][block_size][D]   (token-major inside a block)
 *   V pool: [num_blocks][Hkv][D][block_size]   (channel-major inside a block)
 *   Token slot s lives in block s / block_size at offset s % block_size.
 *   The channel-major V block gives the P.V matrix product its operand with
 *   8 consecutive tokens per 16-byte load.
 * Query / output rows: q and out are [rows][Hq][D]; thread t of a batch owns
 *   the next n_rows[t] rows, in batch order. Row r of thread t sits at context
 *   position L_t - n_rows[t] + r (L_t includes the rows' own tokens) and
 *   attends to positions 0 .. L_t - n_rows[t] + r. Query head h reads KV head
 *   h / (Hq / Hkv). lse is [rows][Hq] float32, natural log.
 */
#ifndef SPORK_H
#define SPORK_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define SPORK_OK 0
#define SPORK_E_INVAL (-1)       /* bad argument (null pointer, bad size, unknown id) */
#define SPORK_E_NOBLOCKS (-2)    /* the free queue cannot serve an append */
#define SPORK_E_UNSUPPORTED (-3) /* dtype / head_dim / block_size without a kernel */
#define SPORK_E_CAPACITY (-4)    /* a caller buffer is too small; required size returned */
#define SPORK_E_HIP (-5)         /* a HIP call or kernel launch failed */

/* ---- element types ----------------------------------------------------- */
#define SPORK_DTYPE_F32 0
#define SPORK_DTYPE_BF16 1

/* Message for the calling thread's last failure ("" if none). Static storage
 * owned by the library, valid until the thread's next failing call. */
const char* spork_last_error(void);

/* ABI version, bumped on any incompatible change. */
int spork_version(void);

/* ======================================================================== *
 *  Block manager (host). Section 4.1: the fork shares the parent's prefix KV.
 * ======================================================================== */
typedef struct spork_cache spork_cache;

/* Create a block manager over num_blocks blocks of block_size tokens.
 * free_order (host, num_blocks entries, nullable): the initial free queue, a
 * permutation of 0..num_blocks-1 taken from the front (NULL = 0,1,2,...).
 * Blocks freed later go to the back of the queue. *out receives the handle,
 * owned by the caller until spork_cache_destroy. */
int spork_cache_create(int32_t num_blocks, int32_t block_size, const int32_t* free_order,
                       spork_cache** out);
int spork_cache_destroy(spork_cache* cache);

/* New empty sequence. Sequence ids are issued 0, 1, 2, ... in creation order
 * (spork_seq_new and spork_fork both create) and are never reused. */
int spork_seq_new(spork_cache* cache, int32_t* seq_out);

/* Reserve slots for n_tokens new tokens at the end of seq.
 * slots_out (host, n_tokens int64): physical slot of each new token.
 * cow_out (host, 3 int32) / n_cow_out: when the sequence ends inside a block
 * that another sequence also references, the first new token makes a private
 * copy: (src_block, dst_block, n_valid) is returned and *n_cow_out = 1; the
 * caller must copy those n_valid slots (spork_kv_copy) before writing the new
 * tokens. Otherwise *n_cow_out = 0. New blocks come from the free queue front;
 * a copy target is taken before any new block. SPORK_E_NOBLOCKS if the queue
 * is too short (nothing changes). */
int spork_seq_append(spork_cache* cache, int32_t seq, int32_t n_tokens, int64_t* slots_out,
                     int32_t* cow_out, int32_t* n_cow_out);

/* Appends to n_seqs distinct sequences (host arrays seqs, n_tokens), in
 * order, with the same result as one spork_seq_append per sequence, for a
 * decode step's bookkeeping in one call. slots_out (host int64, sum of
 * n_tokens entries) receives the slots in batch order; cow_out (host int32,
 * 3 * n_seqs entries) receives *n_cow_out (src, dst, n_valid) copies, in
 * batch order, for spork_kv_copy. All or nothing: the blocks the batch needs
 * are counted first (a copy made unnecessary by an earlier append of the
 * batch is not counted), SPORK_E_NOBLOCKS leaves the cache unchanged;
 * SPORK_E_INVAL for an unknown or repeated sequence or a negative count. */
int spork_seq_append_batch(spork_cache* cache, const int32_t* seqs, const int32_t* n_tokens,
                           int32_t n_seqs, int64_t* slots_out, int32_t* cow_out, int32_t* n_cow_out);

/* Copy-on-write fork (Section 4.1, D1): a new sequence whose table is a copy
 * of parent's; every referenced block gains one reference; no KV is copied. */
int spork_fork(spork_cache* cache, int32_t parent_seq, int32_t* child_seq_out);

/* Drop seq: one reference per table entry in table order; blocks that reach
 * zero references go to the back of the free queue. */
int spork_seq_free(spork_cache* cache, int32_t seq);

int spork_seq_len(const spork_cache* cache, int32_t seq, int32_t* len_out);

/* Block table of seq into out (host, cap entries). *n_out = its length;
 * SPORK_E_CAPACITY (with *n_out set) if cap is too small. */
int spork_block_table(const spork_cache* cache, int32_t seq, int32_t* out, int32_t cap,
                      int32_t* n_out);
int spork_refcount(const spork_cache* cache, int32_t block, int32_t* out);

/* The free queue, front first, into out (host, cap entries); same capacity rule. */
int spork_free_blocks(const spork_cache* cache, int32_t* out, int32_t cap, int32_t* n_out);

/* ======================================================================== *
 *  Shapes and KV writes (setup work around the hot path).
 * ======================================================================== */
typedef struct spork_shape {
  int32_t hq;         /* query heads */
  int32_t hkv;        /* KV heads; hq % hkv == 0 */
  int32_t head_dim;   /* D */
  int32_t block_size; /* tokens per block */
  int32_t dtype;      /* SPORK_DTYPE_*: element type of q, K/V pools and out */
  float sm_scale;     /* softmax scale applied to q.k */
} spork_shape;

/* Write n tokens' K and V into the pools.
 * slots (device, n int64): target slots; k_new, v_new (device, [n][Hkv][D],
 * dtype): the values. Slots outside [0, num_blocks*block_size) are not
 * written and are counted into *bad_slots (device int32, nullable, not
 * cleared by the call). */
int spork_kv_write(const spork_shape* shape, void* k_cache, void* v_cache, int32_t num_blocks,
                   const int64_t* slots, const void* k_new, const void* v_new, int32_t n,
                   int32_t* bad_slots, hipStream_t stream);

/* The copy of copy-on-write: slots 0..n_valid-1 of block src into block dst,
 * every head, both pools (device pools, host arguments). */
int spork_kv_copy(const spork_shape* shape, void* k_cache, void* v_cache, int32_t num_blocks,
                  int32_t src_block, int32_t dst_block, int32_t n_valid, hipStream_t stream);

/* ======================================================================== *
 *  Batch plan (host): the work of one decode / verify step.
 * ======================================================================== */
typedef struct spork_plan spork_plan;

typedef struct spork_plan_info {
  int32_t n_threads;
  int32_t n_rows;          /* query rows (sum of n_rows) */
  int32_t n_groups;        /* fork groups (cascade units) */
  int32_t n_items;         /* (prefix or suffix range, KV head) work items */
  int32_t n_units;         /* attention work units (token range x row slice, incl. padding) */
  int32_t n_partials;      /* partial-result rows written by the attention kernel */
  int32_t max_row_tiles;   /* 16-row MFMA tiles per workgroup */
  int32_t attn_grid;       /* attention workgroups launched */
  size_t image_bytes;      /* size of the device image (spork_plan_image) */
  size_t workspace_bytes;  /* workspace spork_attn_decode needs */
  int64_t shared_tokens;   /* prefix tokens read once per group (sum over groups) */
  int64_t private_tokens;  /* suffix tokens read once per thread */
  int64_t unique_kv_bytes; /* (shared + private tokens) * 2 * Hkv * D * elem */
  int64_t flat_kv_bytes;   /* bytes a kernel without prefix sharing reads */
  int32_t attn_waves;      /* waves per attention workgroup (bf16: 4, two workgroups per
                              compute unit, or 8 when a range has more than 8 row tiles,
                              one per compute unit; fp32: 1) */
  size_t control_bytes;    /* leading workspace bytes that hold control words (see
                              spork_workspace_clear) */
} spork_plan_info;

/* Plan one step for n_threads threads.
 * seqs, n_rows, groups (host, n_threads each): the sequences, their query
 * rows (1 for decode, K+1 for a verify thread; 1 <= n_rows <= length) and
 * their fork group (threads with the same group id >= 0 share their longest
 * common block-table prefix; -1 = no group). n_cu: compute units to balance
 * for (0 = 256, one MI355X). The plan keeps no reference to the cache. */
int spork_plan_create(const spork_cache* cache, const spork_shape* shape, const int32_t* seqs,
                      const int32_t* n_rows, const int32_t* groups, int32_t n_threads,
                      int32_t n_cu, spork_plan** out);
int spork_plan_destroy(spork_plan* plan);
int spork_plan_get_info(const spork_plan* plan, spork_plan_info* info);

/* Reuse a plan for a later decode step (Sections 4.1 and 4.3: every main
 * and probe thread keeps decoding; the batch stays the same).
 * After tokens were appended to the plan's threads (spork_seq_append on
 * `cache`, the cache the plan was made from), bring the plan and its device
 * image up to the threads' current lengths: each thread's private range
 * (the part of its context no other thread of its group shares), its rows'
 * positions (still the last n_rows[t] positions of the context) and its
 * block table grow with it. The work split is kept, so this costs
 * O(threads + new blocks) host time and, when anything changed, one small
 * kernel on `stream` per 480 changed words of `dev_image` (the device copy
 * of spork_plan_image, 256-byte aligned; the patch travels in the kernel's
 * arguments, nothing is copied from the host). Call it after the appends
 * and before the step's attention call, on the same stream.
 * SPORK_E_CAPACITY when the plan cannot absorb the growth: more new blocks
 * than the 64 the image reserves per thread table, a private range past
 * the longest unit the kernel stages, or a grown thread with no private
 * range; SPORK_E_INVAL when a planned sequence was freed, shrank or had a
 * planned block replaced (copy-on-write). In both cases nothing is launched,
 * the plan is unchanged, and the caller plans again. */
int spork_plan_advance(spork_plan* plan, const spork_cache* cache, void* dev_image,
                       hipStream_t stream);

/* Copy the plan's device image (block tables, work list, merge lists) into
 * host_dst (cap bytes, >= info.image_bytes). The caller places it in device
 * memory (256-byte aligned) and passes that copy as dev_image below. */
int spork_plan_image(const spork_plan* plan, void* host_dst, size_t cap);

/* ======================================================================== *
 *  Hot path.
 * ======================================================================== */

/* Workspace control words. The first info.control_bytes bytes of a plan's
 * workspace are the work-list cursors of the persistent bf16 attention
 * launch. They must be zero when a call starts, and every call leaves them
 * zero (its last launch clears them). Zero them once after allocating a workspace, and again
 * before a workspace serves a plan with a larger control_bytes than the
 * plans it served before (bytes past the old control words held partial
 * results): this call does it with one small kernel on `stream` (no
 * memset, so it may be captured in a HIP graph). ws_bytes >=
 * info.control_bytes; the rest of the workspace is not touched. */
int spork_workspace_clear(const spork_plan* plan, void* workspace, size_t ws_bytes,
                          hipStream_t stream);

/* Batched decode attention of main and probe rows (Sections 4.1 and 4.3).
 * q (device [rows][Hq][D] dtype); k_cache, v_cache (device pools);
 * out (device [rows][Hq][D] dtype); lse (device [rows][Hq] float32, nullable);
 * workspace (device, 256-byte aligned, ws_bytes >= info.workspace_bytes;
 * control words zero on entry, see spork_workspace_clear, the rest any
 * contents; it holds the partial results and the counters, so calls that
 * share a workspace must not overlap).
 * Two launches on `stream`: the partial attention over prefix and suffix
 * ranges (bf16: persistent workgroups working through per-compute-unit
 * lists), then the log-sum-exp merge, which also returns the cursors to
 * zero. */
int spork_attn_decode(const spork_plan* plan, const void* dev_image, const void* q,
                      const void* k_cache, const void* v_cache, void* out, float* lse,
                      void* workspace, size_t ws_bytes, hipStream_t stream);

/* Workspace for the argmax + accept part of spork_verify_accept. */
int spork_verify_workspace_bytes(int32_t n_verify, int32_t k_drafts, int32_t vocab,
                                 size_t* bytes);

/* D3 verify step (Section 4.3): optional attention over the plan (pass
 * plan = NULL to run only the accept), then greedy argmax over the verify
 * logits and the longest-prefix accept.
 * logits (device [n_verify*(k_drafts+1)][vocab], logits_dtype): row
 * s*(k_drafts+1)+r is verify row r of verify thread s; drafts (device
 * [n_verify][k_drafts] int32). Outputs (device int32): accept_len[n_verify]
 * = first r < k_drafts whose greedy token differs from the draft, else
 * k_drafts; next_token[n_verify] = greedy token of row accept_len;
 * argmax_out[n_verify*(k_drafts+1)] (nullable) = every row's greedy token.
 * Ties pick the lowest vocabulary index; logits must be finite. A draft of
 * -1 (padding after fewer than k_drafts real drafts) never matches.
 * workspace: the attention's workspace followed (at a 256-byte aligned
 * offset) by spork_verify_workspace_bytes; ws_bytes covers both. With a
 * plan the workspace's control words must be zero on entry
 * (spork_workspace_clear).
 * With a bf16 plan the step is two launches on `stream`: the partial
 * attention, whose persistent workgroups take the argmax units once their
 * own lists are done, then the merge together with the accept (and the
 * cursor clear). fp32 plan: the argmax, the partial attention, the merge
 * with the accept. Without a plan: the argmax, then the accept. */
int spork_verify_accept(const spork_plan* plan, const void* dev_image, const void* q,
                        const void* k_cache, const void* v_cache, void* out, float* lse,
                        const void* logits, int32_t logits_dtype, int32_t vocab,
                        const int32_t* drafts, int32_t n_verify, int32_t k_drafts,
                        int32_t* accept_len, int32_t* next_token, int32_t* argmax_out,
                        void* workspace, size_t ws_bytes, hipStream_t stream);

/* spork_verify_accept without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation). Same arguments and results as
 * spork_verify_accept (plan may be NULL, n_verify may be 0), same kernels;
 * the partial results, cursors and argmax keys live in a library-owned
 * 64 MiB array per GPU (a device global, held until the process ends)
 * instead of the workspace. A step that needs more (the sum of
 * info.workspace_bytes rounded up to 256 and spork_verify_workspace_bytes)
 * is rejected with SPORK_E_CAPACITY before anything is launched; use
 * spork_verify_accept for it. No device memory is allocated or freed and
 * no timing events are recorded. The first call on a device looks up that
 * device's array; a call whose plan needs more zeroed control words than
 * the previous call left zero launches a small clearing kernel first.
 * Every call on one GPU shares that GPU's array, which keeps the last
 * call's contents: calls that overlap on one GPU (different streams or
 * threads) race and must be serialised by the caller. */
int spork_verify_accept_noalloc(const spork_plan* plan, const void* dev_image, const void* q,
                                const void* k_cache, const void* v_cache, void* out, float* lse,
                                const void* logits, int32_t logits_dtype, int32_t vocab,
                                const int32_t* drafts, int32_t n_verify, int32_t k_drafts,
                                int32_t* accept_len, int32_t* next_token, int32_t* argmax_out,
                                hipStream_t stream);

/* Workspace for spork_probe_confidence. */
int spork_confidence_workspace_bytes(int32_t n_rows, int32_t vocab, size_t* bytes);

/* D2 confidence gate (Section 4.2, confidence score).
 * logits (device [n_rows][vocab], logits_dtype f32 or bf16): one row per
 * generated probe position; every row needs a finite maximum (-inf entries
 * are allowed, NaN is not). span_off (device int32 [n_probes+1],
 * non-decreasing, within [0, n_rows]): probe p's tool-name span is rows
 * span_off[p] .. span_off[p+1]-1; offsets are clamped to [0, n_rows] and a
 * reversed span counts as empty, so bad offsets never read out of bounds.
 * Outputs (device): argmax_out[n_rows] int32 (nullable) = greedy token, the
 *   lowest index of the row maximum; logprob_out[n_rows] float32 (nullable)
 *   = top-1 log-probability max(x) - ln(sum exp(x)), accumulated in float32;
 *   confidence_out[n_probes] float32 = min over the span's rows after the
 *   first of exp(logprob), 1.0 for a span of fewer than two rows;
 *   commit_out[n_probes] int32 (nullable) = confidence_out >= theta, decided
 *   in float32.
 * workspace (device, 256-byte aligned, ws_bytes >= the size from
 * spork_confidence_workspace_bytes; any contents on entry).
 * Two launches on `stream`: per-chunk argmax and sum of exponentials, then
 * per-row results and the per-probe gate. SPORK_E_INVAL for bad sizes or a
 * NULL required pointer, SPORK_E_UNSUPPORTED for another logits dtype,
 * SPORK_E_CAPACITY for a short workspace. */
int spork_probe_confidence(const void* logits, int32_t logits_dtype, int32_t vocab,
                           int32_t n_rows, const int32_t* span_off, int32_t n_probes,
                           float theta, int32_t* argmax_out, float* logprob_out,
                           float* confidence_out, int32_t* commit_out, void* workspace,
                           size_t ws_bytes, hipStream_t stream);

/* Workspace for spork_ngram_propose. */
int spork_ngram_workspace_bytes(int32_t n_seqs, int64_t max_len, size_t* bytes);

/* n-gram (prompt-lookup) drafts for a batch of token sequences: the baseline
 * draft source of the paper's engine configuration (Section 6.1), which D3's
 * proposer wraps (Section 4.3).
 * tokens (device int32): the sequences (prompt and output so far) one after
 * another; seq_off (device int64 [n_seqs+1]): sequence s is tokens
 * seq_off[s] .. seq_off[s+1]-1 (offsets non-decreasing, within the tokens
 * buffer, each sequence shorter than 2^31 tokens; they are read on the
 * device and not checked).
 * For each sequence of L tokens: for n from n_max down to n_min, the key is
 * its last n tokens; the first n whose key occurs earlier, starting at j
 * with j + n <= L - 1 (occurrences may overlap the key), wins, and of its
 * occurrences the latest. The drafts are the up to k tokens after that
 * occurrence, cut at the end of the sequence.
 * Outputs (device int32): drafts[n_seqs][k], -1 past n_drafts[s] (a value
 * no greedy token takes, so spork_verify_accept accepts at most the real
 * drafts); n_drafts[n_seqs] in [0, k].
 * max_len sizes the launch (one workgroup per 2048 positions of the longest
 * sequence expected); longer sequences are still scanned whole, more slowly.
 * workspace (device, 256-byte aligned, ws_bytes >= the size from
 * spork_ngram_workspace_bytes; any contents on entry).
 * Two launches on `stream`. SPORK_E_INVAL for bad sizes (1 <= n_min <=
 * n_max <= 32, 0 <= k <= 4096, 0 <= max_len < 2^31) or a NULL required
 * pointer, SPORK_E_CAPACITY for a short workspace. */
int spork_ngram_propose(const int32_t* tokens, const int64_t* seq_off, int32_t n_seqs,
                        int64_t max_len, int32_t n_min, int32_t n_max, int32_t k,
                        int32_t* drafts, int32_t* n_drafts, void* workspace, size_t ws_bytes,
                        hipStream_t stream);

/* ======================================================================== *
 *  Kernel timing (benchmarks).
 * ======================================================================== */
#define SPORK_KERNEL_ATTN 0   /* cascade / private-range partial attention */
#define SPORK_KERNEL_MERGE 1  /* log-sum-exp merge (+ the verify step's accept) */
#define SPORK_KERNEL_ARGMAX 2 /* greedy argmax over vocabulary chunks */
#define SPORK_KERNEL_ACCEPT 3 /* accept of an accept-only call (plan == NULL) */
#define SPORK_KERNEL_CONF_CHUNKS 4 /* confidence: per-chunk argmax and sum of exponentials */
#define SPORK_KERNEL_CONF_FINAL 5  /* confidence: per-row log-probability and per-probe gate */
#define SPORK_KERNEL_NGRAM_SCAN 6  /* n-gram drafts: per-chunk longest latest key match */
#define SPORK_KERNEL_NGRAM_DRAFTS 7 /* n-gram drafts: per-sequence choice and draft copy */
#define SPORK_KERNEL_READ_CEILING 8 /* streaming-read ceiling (measurement aid) */
#define SPORK_KERNEL_KINDS 9

/* Streaming-read ceiling (a measurement aid, not a step of the method): read
 * `bytes` of the device buffer `src` once, with `grid` workgroups of 256
 * threads, each taking a contiguous share. It gives the bandwidth a plain
 * read stream reaches on this device, the ceiling the attention launch is
 * compared with.
 *   mode 0: 16-byte register loads, 8 in flight per thread;
 *   mode 1: direct-to-LDS loads in the bf16 attention kernel's ring shape
 *           (4 waves, 4 slots of 16 KB, 3 in flight) with no arithmetic;
 *           bytes must be a multiple of grid * 16384;
 *   mode 2: as mode 0 with non-temporal loads;
 *   mode 3: as mode 1 with non-temporal loads (same bytes rule).
 * sink (device, caller-owned): grid * 256 uint32 words, overwritten with
 * XOR folds of the data (so no load is dead). src 16-byte aligned, bytes a
 * positive multiple of 16, 1 <= grid <= 65536; otherwise SPORK_E_INVAL and
 * nothing is launched. One launch on `stream`. */
int spork_read_ceiling(const void* src, int64_t bytes, int32_t grid, int32_t mode, uint32_t* sink,
                       hipStream_t stream);

/* While enabled (per calling thread), every hot-path call records a HIP event
 * before and after each of its kernels on the caller's stream. */
int spork_timing_enable(int32_t on);

/* Wait for the recorded events, write the summed milliseconds and the launch
 * count of each kernel kind into ms_out / launches_out (host arrays of
 * SPORK_KERNEL_KINDS entries, launches_out nullable), and start a new
 * accumulation. SPORK_E_HIP if an event cannot be read. */
int spork_timing_read(float* ms_out, int32_t* launches_out);

#ifdef __cplusplus
}
#endif
#endif /* SPORK_H */
