/*
 * tts.h -- C ABI of libtts: decode-step attention for test-time-scaling
 * beam search over a paged KV cache whose blocks are shared along the beams'
 * common prefixes.
 *
 * Problem (FastTTS, Sec. 3.1 and Sec. 4.2): a verifier-guided search keeps N
 * reasoning beams per request; every decode step each beam issues one query
 * token that attends over its own cached keys/values. Beams duplicated from
 * one parent share that parent's KV blocks, so the beams of a request form a
 * radix tree (trie) of shared prefixes. Decoding is memory-bandwidth bound
 * (Sec. 3.2.3), so the library reads every shared block once per group of
 * beams that shares it instead of once per beam.
 *
 * Conventions shared by every call
 * --------------------------------
 * - Status: every call returns tts_status; TTS_OK (0) on success, a negative
 *   code otherwise. tts_last_error() returns a thread-local message for the
 *   last failing call of the calling thread. Nothing throws or exits.
 * - Ownership: the library never allocates or frees caller buffers. Device
 *   pointers (q, caches, scales, tables, lengths, out, workspace) are owned
 *   by the caller and must stay valid until the enqueued work completes.
 *   A tts_prefix_meta handle owns host arrays and one device buffer; free it
 *   with tts_prefix_meta_destroy.
 * - Asynchrony: device calls validate their host-visible arguments, enqueue
 *   kernels on `stream` and return; kernel faults surface at the caller's
 *   next synchronisation. Calls keep no global state and are reentrant;
 *   concurrent calls must use distinct workspaces.
 * - Layouts (row-major, element strides implied by the shapes):
 *     q          [num_seqs][Hq][D]                     (F32 or BF16)
 *     k_cache    [num_blocks][Hkv][block_size][D]      token-major blocks
 *     v_cache    [num_blocks][Hkv][D][block_size]      dim-major blocks
 *     k_scale, v_scale [num_blocks] fp32               (FP8 caches only)
 *     block_tables [num_seqs][max_blocks_per_seq] int32 physical block ids
 *     seq_lens   [num_seqs] int32
 *     out        [num_seqs][Hq][D] fp32
 * - Semantics (Sec. 3.1 generation step): seq_lens[b] counts the cached
 *   tokens of beam b including the current one (its K/V are already in the
 *   cache). Query head h uses KV head h / (Hq / Hkv). The result is
 *   softmax(scale * q K^T) V over the beam's seq_lens[b] tokens; a beam with
 *   seq_len 0 gets a zero row. Table entries at or past
 *   ceil(seq_len / block_size) are never read, and neither are the unused
 *   slots of a partially filled last block.
 * - FP8 KV: OCP E4M3FN codes; the value of a code in block p is
 *   decode(code) * k_scale[p] (keys) or * v_scale[p] (values).
 * - Device-side errors: a block id outside [0, num_blocks) read from a
 *   device table (any entry in the paged call; an entry appended after the
 *   metadata was built in the prefix call -- entries in use at build time
 *   are validated by tts_build_prefix_meta), a sequence longer than its
 *   table row, or (prefix call) a beam shorter than the metadata was built
 *   for makes that beam's output row NaN; no memory outside the given
 *   buffers is touched.
 */
#ifndef TTS_H_
#define TTS_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TTS_OK = 0,
  TTS_ERR_INVALID_ARG = -1,
  TTS_ERR_UNSUPPORTED = -2,
  TTS_ERR_OUT_OF_RANGE = -3,
  TTS_ERR_WORKSPACE = -4,
  TTS_ERR_HIP = -5,
  TTS_ERR_NOMEM = -6
} tts_status;

typedef enum { TTS_F32 = 0, TTS_BF16 = 1, TTS_FP8_E4M3 = 2 } tts_dtype;

/* Attention shape. Supported: Hq % Hkv == 0, head_dim 64 or 128,
 * block_size 16; (q, kv) dtypes (F32, F32), (BF16, BF16), (BF16, FP8_E4M3);
 * out_dtype F32. scale <= 0 selects 1/sqrt(head_dim). */
typedef struct {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t block_size;
  tts_dtype q_dtype;
  tts_dtype kv_dtype;
  tts_dtype out_dtype;
  float scale;
} tts_attn_desc;

/* Opaque prefix metadata of one batch of requests (host arrays + one device
 * buffer with the kernels' work list). */
typedef struct tts_prefix_meta tts_prefix_meta;

/* Canonical view of the metadata (host pointers, valid until destroy).
 * perm[i]: original index of the beam at position i. Segments are maximal
 * chains of trie nodes with the same set of >= 2 beams, listed in depth-first
 * preorder; segment s covers logical blocks [seg_lblock_begin[s],
 * seg_lblock_begin[s] + seg_nblocks[s]) of the beams at positions
 * [seg_beam_begin[s], seg_beam_end[s]) of perm; seg_parent[s] is the
 * enclosing segment or -1. tail_lblock[b] (original index b) is the first
 * logical block of beam b not covered by a segment. unique_blocks counts
 * the distinct physical ids in use; unique_tokens sums, over those ids, the
 * largest number of valid tokens any beam sees in the block. */
typedef struct {
  int32_t num_seqs;
  int32_t num_segs;
  const int32_t* perm;
  const int32_t* seg_req;
  const int32_t* seg_parent;
  const int32_t* seg_lblock_begin;
  const int32_t* seg_nblocks;
  const int32_t* seg_beam_begin;
  const int32_t* seg_beam_end;
  const int32_t* tail_lblock;
  int64_t unique_blocks;
  int64_t unique_tokens;
} tts_prefix_meta_view;

/* Build the prefix metadata of a batch (Sec. 4.2: the beams of each request
 * form a radix tree of shared thinking prefixes; beams spawned from the same
 * parent are grouped while the parents keep their relative order).
 *
 * All array arguments are HOST int32 arrays; they are copied, not retained.
 *   req_seq_offsets [num_reqs + 1]: CSR offsets of each request's beams,
 *       offsets[0] == 0, non-decreasing, offsets[num_reqs] == num_seqs.
 *   block_tables [num_seqs * max_blocks_per_seq], seq_lens [num_seqs].
 * Per request, a trie is built over each beam's FULL blocks
 * (seq_len / block_size of them); only blocks whose id and every preceding
 * id agree are shared; partial last blocks and blocks of different requests
 * are never shared. Children are ordered by the smallest original beam index
 * they contain.
 * desc: if non-NULL, the kernels' work list for this attention shape is
 *   built and uploaded to a device buffer on `stream` (the handle can then
 *   be passed to tts_prefix_decode_attn with the same desc); if NULL, only
 *   the host-side metadata is built (export/coverage only, no device use).
 * Errors: TTS_ERR_INVALID_ARG (bad offsets, lengths, sizes, NULL pointers),
 *   TTS_ERR_OUT_OF_RANGE (a block id in use outside [0, num_blocks)),
 *   TTS_ERR_UNSUPPORTED (desc shape), TTS_ERR_HIP, TTS_ERR_NOMEM. */
tts_status tts_build_prefix_meta(int32_t num_reqs, const int32_t* req_seq_offsets, int32_t num_seqs,
                                 const int32_t* block_tables, int32_t max_blocks_per_seq,
                                 const int32_t* seq_lens, int32_t block_size, int32_t num_blocks,
                                 const tts_attn_desc* desc, hipStream_t stream, tts_prefix_meta** out);

/* The metadata of a batch after a fork (Sec. 3.1, Alg. 1: survivors are
 * duplicated, each iteration's schedule is fixed once, Sec. 4.2), built from
 * the previous batch's handle: the trie, segments and beam order are built
 * for the new tables as tts_build_prefix_meta builds them (bit for bit), and
 * the work plan starts from prev's target unit cost, scaled by the change in
 * total work, instead of searching for one (the search is most of a full
 * build's host time). The desc is prev's. Arguments, errors and result as in
 * tts_build_prefix_meta (the plan may differ from the one a full build
 * picks; attention results agree to rounding). prev: built with a desc, not
 * a verification metadata; it stays valid and owned by the caller. */
tts_status tts_fork_prefix_meta(const tts_prefix_meta* prev, int32_t num_reqs, const int32_t* req_seq_offsets,
                                int32_t num_seqs, const int32_t* block_tables, int32_t max_blocks_per_seq,
                                const int32_t* seq_lens, int32_t block_size, int32_t num_blocks, hipStream_t stream,
                                tts_prefix_meta** out);

/* Free a handle (NULL is ignored). The device buffer is released with
 * hipFree, which waits for work still using it. */
void tts_prefix_meta_destroy(tts_prefix_meta* m);

/* Fill `view` with host pointers into the handle's canonical arrays. */
tts_status tts_prefix_meta_export(const tts_prefix_meta* m, tts_prefix_meta_view* view);

/* Indexing export: one row (beam, lblock, pblock, ntok, src) per used
 * (beam, logical block), beams in original order and each beam's blocks in
 * merge order (segments root to leaf, then the tail); src is the covering
 * segment or -1 for tail blocks. seq_lens_host (may be NULL: build-time
 * lengths) may exceed the build-time lengths (private appends); pblock of
 * such rows comes from the tables as given at build time. out_rows holds
 * cap rows of 5 int32; *n_rows receives the number of rows needed.
 * TTS_ERR_WORKSPACE if cap is too small (n_rows still set). */
tts_status tts_prefix_meta_coverage(const tts_prefix_meta* m, const int32_t* seq_lens_host, int32_t* out_rows,
                                    int64_t cap, int64_t* n_rows);

/* Work-list statistics of a handle built with a desc: number of kernel work
 * units and partial-result slots (for diagnostics and benchmarks). */
tts_status tts_prefix_meta_stats(const tts_prefix_meta* m, int64_t* num_units, int64_t* num_slots);

/* Host-only inspection of the work plan (no device is touched): the plan
 * tts_build_prefix_meta makes for this desc when the device has
 * num_workgroups compute units (one persistent workgroup each), listed as
 * one row per (unit, block entry, beam the entry applies to), 7 int32:
 *   {unit, entry, kv_head, beam, block, valid, flags}
 * unit numbers the units with work; entry counts across the unit's windows;
 * beam is the original beam index; block the physical block id (-1 for an
 * extension entry: the beam's blocks appended after the build, read from
 * the live table at call time); valid its build-time token count (0 for
 * extension entries). flags: 1 = the beam's partially filled last block
 * (its valid count follows the live length), 2 = extension entry,
 * 4 = in the unit's second window, 8 = wide unit (LDS-staged blocks that
 * apply to all its rows). Arguments as in tts_build_prefix_meta, which
 * validates them the same way. out_rows holds cap rows; *n_rows receives
 * the number of rows needed and *num_units the number of units (also when
 * cap is too small: TTS_ERR_WORKSPACE). For tests and diagnostics. */
tts_status tts_plan_units_host(int32_t num_reqs, const int32_t* req_seq_offsets, int32_t num_seqs,
                               const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                               int32_t block_size, int32_t num_blocks, const tts_attn_desc* desc,
                               int32_t num_workgroups, int32_t* out_rows, int64_t cap, int64_t* n_rows,
                               int64_t* num_units);

/* Workspace bytes needed by tts_paged_decode_attn for these sizes. */
size_t tts_paged_decode_workspace_size(const tts_attn_desc* d, int32_t num_seqs, int32_t max_seq_len);

/* Decode attention of every beam over its own paged sequence, without
 * exploiting sharing: every beam reads all of its blocks (the non-sharing
 * baseline; paged attention of the serving substrate, Sec. 2.3).
 * max_seq_len: host upper bound on seq_lens (sizes the split of long
 * sequences); beams longer than it get NaN rows.
 * num_blocks: size of the block pool (ids outside it give NaN rows).
 * workspace: device buffer of at least tts_paged_decode_workspace_size
 * bytes (TTS_ERR_WORKSPACE otherwise); NULL allowed when that size is 0.
 * Calls that overlap in time must not share a workspace. More than
 * 2^31 - 1 partial rows (num_seqs x splits x query heads) is
 * TTS_ERR_UNSUPPORTED. */
tts_status tts_paged_decode_attn(const tts_attn_desc* d, int32_t num_seqs, const void* q, const void* k_cache,
                                 const void* v_cache, const float* k_scale, const float* v_scale,
                                 const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                 int32_t max_seq_len, int32_t num_blocks, void* out, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes needed by tts_prefix_decode_attn with this metadata. */
size_t tts_prefix_decode_workspace_size(const tts_attn_desc* d, const tts_prefix_meta* m);

/* Prefix-shared decode attention (Sec. 4.2 prefix sharing applied to the
 * decode step): each shared segment's KV blocks are read once per group of
 * beams sharing them and staged in LDS for all of that group's query rows;
 * each beam's private tail is read by that beam alone; the pieces are
 * combined by an exact log-sum-exp merge in a fixed order. Same result as
 * tts_paged_decode_attn up to rounding.
 * m: built with the same desc shape and with the same block tables, and
 * still valid: every table entry in use at build time is unchanged and
 * every seq_len is >= its value at build time (beams only appended
 * privately). The ids of the blocks in use at build time are taken from
 * the metadata; blocks appended since are read from block_tables.
 * block_tables/seq_lens: device copies of the current tables and lengths.
 * workspace: at least tts_prefix_decode_workspace_size bytes (partial
 * softmax states; calls that overlap in time must not share one). A plan
 * with more than 2^31 - 1 partial rows is TTS_ERR_UNSUPPORTED. */
tts_status tts_prefix_decode_attn(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q,
                                  const void* k_cache, const void* v_cache, const float* k_scale,
                                  const float* v_scale, const int32_t* block_tables, int32_t max_blocks_per_seq,
                                  const int32_t* seq_lens, int32_t num_blocks, void* out, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 * tts_prefix_decode_attn without a workspace argument; arguments, rules and
 * results are those of tts_prefix_decode_attn (same kernels, same plan).
 * The partial softmax states go to a scratch array of 64 MiB that the
 * library holds on each GPU it runs on, from the first call on that GPU
 * until the process ends; nothing is allocated or freed (no hipMalloc,
 * hipFree or allocating library call). A metadata whose
 * tts_prefix_decode_workspace_size exceeds 64 MiB is refused with
 * TTS_ERR_WORKSPACE before anything is enqueued. Every call on one GPU uses
 * that GPU's one array: calls that overlap in time on the same GPU (two
 * streams, or two host threads) race on it and must be serialised by the
 * caller. */
tts_status tts_prefix_decode_attn_noalloc(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q,
                                          const void* k_cache, const void* v_cache, const float* k_scale,
                                          const float* v_scale, const int32_t* block_tables,
                                          int32_t max_blocks_per_seq, const int32_t* seq_lens, int32_t num_blocks,
                                          void* out, hipStream_t stream);

/* ---- Verification attention over the shared prefix (LookAhead
 * Verification, Sec. 4.1: the current and the speculative step go to the
 * verifier as one request; its attention is a multi-token causal attention
 * over each path's shared prefix). Every beam's last q_len cached tokens are
 * queries: query i of beam b (position seq_lens[b] - q_len + i) attends to
 * the beam's tokens 0 .. seq_lens[b] - q_len + i (causal). The metadata
 * (tts_build_verify_meta) treats query i of beam b as a virtual beam
 * b * q_len + i whose length ends at that position, so the shared blocks are
 * read once for every query row of every beam that shares them.
 * tts_build_verify_meta: as tts_build_prefix_meta, plus q_len >= 1; every
 * seq_len must be >= q_len. Exported views and coverage rows describe the
 * virtual beams. */
tts_status tts_build_verify_meta(int32_t num_reqs, const int32_t* req_seq_offsets, int32_t num_seqs,
                                 const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                 int32_t q_len, int32_t block_size, int32_t num_blocks, const tts_attn_desc* desc,
                                 hipStream_t stream, tts_prefix_meta** out);

/* q: [num_seqs][q_len][Hq][D], out: [num_seqs][q_len][Hq][D] fp32;
 * block_tables [num_seqs][max_blocks_per_seq] and seq_lens [num_seqs] are
 * the beams' own (device); the other arguments and rules are those of
 * tts_prefix_decode_attn (which refuses a verification metadata). The
 * partials/merge pair below also accepts a verification metadata. */
tts_status tts_prefix_verify_attn(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q,
                                  const void* k_cache, const void* v_cache, const float* k_scale,
                                  const float* v_scale, const int32_t* block_tables, int32_t max_blocks_per_seq,
                                  const int32_t* seq_lens, int32_t num_blocks, void* out, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);

/* The two launches of tts_prefix_decode_attn, for callers that schedule
 * them separately (to overlap the merge with other work, or to time the
 * attention kernel alone). tts_prefix_decode_partials runs the work units
 * and leaves one partial softmax state (reference max, sum, and the output
 * row: for bf16 and fp8 caches in fp16, divided by a power of two, with a
 * factor that takes it to the row normalised by the sum; for fp32 caches
 * normalised, in fp32) per (beam, query head, slot) in the workspace;
 * tts_prefix_decode_merge combines each beam's states, in slot order, into
 * out. Arguments and rules are those of tts_prefix_decode_attn; the merge
 * must follow the partials call on the same workspace in stream order, with
 * the same metadata and seq_lens. */
tts_status tts_prefix_decode_partials(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q,
                                      const void* k_cache, const void* v_cache, const float* k_scale,
                                      const float* v_scale, const int32_t* block_tables,
                                      int32_t max_blocks_per_seq, const int32_t* seq_lens, int32_t num_blocks,
                                      void* out, void* workspace, size_t workspace_bytes, hipStream_t stream);
tts_status tts_prefix_decode_merge(const tts_attn_desc* d, const tts_prefix_meta* m, const int32_t* seq_lens,
                                   void* out, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ---- KV-cache maintenance around the decode step ---------------------------
 *
 * A decode step writes each beam's new token into the paged cache before the
 * attention reads it (seq_len counts it), and the search's duplication step
 * (DuplicateThenTruncate, Sec. 3.1 and Alg. 1: surviving beams are
 * duplicated; the duplicates' speculative tokens are truncated, Sec. 4.1)
 * shares a parent's full blocks with its children and copies the partially
 * filled block each child keeps (copy-on-write). */

/* Append: for every beam b with L = seq_lens[b] > 0, store its token at
 * position L - 1 (slot (L - 1) % 16 of block block_tables[b][(L - 1) / 16]):
 * k_new[b][h][:] into that block's K row of KV head h, v_new[b][h][:] into
 * its V column. k_new, v_new: [num_seqs][Hkv][D] device arrays, bf16 for
 * BF16 and FP8_E4M3 caches, fp32 for F32 caches. Beams with seq_len 0, a
 * block index past their table row or a block id outside [0, num_blocks)
 * write nothing.
 * FP8 caches (k_scale/v_scale required): each of K and V is stored as
 * E4M3FN codes of value / scale[block] (round to nearest even, saturating
 * at 448). A token opening a block (slot 0) sets the block's scale to
 * amax / 448 over the token's values of all KV heads (1 if all are zero);
 * a later token whose amax exceeds 448 * scale raises the scale to
 * amax / 448 and re-encodes the block's earlier codes of every head under
 * it (decode * old scale / new scale); otherwise the scale is kept.
 * Every beam's current block must belong to that beam alone (a shared
 * partial block is copied first, see tts_fork_tables); beams writing the
 * same block in one call race. */
tts_status tts_append_kv(const tts_attn_desc* d, int32_t num_seqs, const void* k_new, const void* v_new,
                         const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                         int32_t num_blocks, void* k_cache, void* v_cache, float* k_scale, float* v_scale,
                         hipStream_t stream);

/* Copy whole blocks: for each i < num_pairs, K and V of every KV head of
 * block pairs[2i] into block pairs[2i + 1] (and the fp8 scales). pairs is a
 * device int32 array. Pairs naming a block outside [0, num_blocks), or a
 * block onto itself, copy nothing. Destinations must be distinct and not
 * be sources of the same call. */
tts_status tts_copy_blocks(const tts_attn_desc* d, int32_t num_pairs, const int32_t* pairs, int32_t num_blocks,
                           void* k_cache, void* v_cache, float* k_scale, float* v_scale, hipStream_t stream);

/* Host: block tables of duplicated beams. Child c copies the first
 * child_lens[c] tokens of beam child_parent[c] (0 <= child_lens[c] <=
 * parent length; a shorter child drops its parent's speculative tokens).
 * Its full blocks are its parent's (shared, same ids); a partially filled
 * last block becomes the next id of free_ids, and the pair (parent's
 * block, new id) is appended to copies ([num_children][2] capacity) for
 * tts_copy_blocks. Entries past the child's blocks are -1. All arrays are
 * host int32: parent_tables [num_parents][max_blocks_per_seq],
 * child_tables [num_children][max_blocks_per_seq] (written). Outputs the
 * number of copies and of free ids consumed (in order). Errors
 * (TTS_ERR_OUT_OF_RANGE for a bad parent index, TTS_ERR_INVALID_ARG for a
 * bad length, TTS_ERR_NOMEM when free_ids runs out) are detected before
 * anything is written. */
tts_status tts_fork_tables(int32_t num_parents, const int32_t* parent_tables, int32_t max_blocks_per_seq,
                           const int32_t* parent_lens, int32_t block_size, int32_t num_children,
                           const int32_t* child_parent, const int32_t* child_lens, const int32_t* free_ids,
                           int32_t num_free, int32_t* child_tables, int32_t* copies, int32_t* num_copies,
                           int32_t* num_free_used);

/* Host: lengths of duplicated beams after speculation (Sec. 4.1, Alg. 1
 * DuplicateThenTruncate: only the duplicates of a speculated beam lose
 * speculative tokens, the original stays whole; the truncation is drawn from
 * a normal distribution with mean R, the truncation ratio). Children are
 * listed as for tts_fork_tables (child_parent[c] in [0, num_parents)); the
 * first child of each parent is its original and keeps parent_lens[p]
 * tokens; every later child of p keeps the parent's first
 * parent_lens[p] - parent_spec[p] tokens plus
 * floor(clip(ratio + sigma z[c], 0, 1) * parent_spec[p] + 0.5) of its
 * parent_spec[p] speculative ones (the product sigma z[c] and the one with
 * parent_spec rounded to double before the sums). z: one standard-normal
 * draw per child (the caller's generator; entries of originals unused).
 * The paper leaves the spread open (sigma = 0.1 is the reading the tests
 * use). Writes child_lens[num_children] for tts_fork_tables.
 * Errors (before anything is written): TTS_ERR_OUT_OF_RANGE for a bad parent,
 * TTS_ERR_INVALID_ARG for parent_spec outside [0, parent length], a
 * non-finite ratio or z, or sigma < 0. */
tts_status tts_truncated_lengths(int32_t num_children, const int32_t* child_parent, const int32_t* parent_lens,
                                 const int32_t* parent_spec, int32_t num_parents, double ratio, double sigma,
                                 const double* z, int32_t* child_lens);

/* ---- Roofline-guided KV allocation (Sec. 4.3) -------------------------------
 *
 * Split one KV-cache budget M between the verifier (prefill) and the
 * generator (decode) to minimise the modelled total time of N requests:
 *   T_tot = ceil(N / B_pre) * T_pre(B_pre, S)
 *         + ceil(N / B_dec) * S_dec * T_dec(B_dec, S_dec / 2)
 * subject to B_pre * KV_v(S) + B_dec * KV_g(S_dec) <= M, with
 * T = max(FLOPs / peak_flops, bytes / peak_bw) per batch (roofline). For a
 * model m: a prefill of b sequences of s tokens costs 2 params b s +
 * 2 L d b s (s + 1) flops (dense layers; causal attention) and
 * weight_bytes + b kv s bytes (weights read once, KV written); a decode step
 * of b sequences over c cached tokens costs 2 params b + 4 L d b c flops
 * and weight_bytes + b kv c bytes (KV read); KV_m(s) = kv_bytes_per_token s.
 * The search tries every prefill batch 1 <= B_pre <= N that leaves room for
 * one decode sequence, with the decode batch on the memory boundary,
 * B_dec = min(N, floor((M - B_pre KV_v(S)) / KV_g(S_dec))), and keeps the
 * fastest pair, ties going to the larger B_dec. (Batches are capped at N:
 * a batch never holds more requests than there are.) Host calls. */
typedef struct {
  double params;             /* parameter count */
  double weight_bytes;       /* bytes of weights read per forward pass */
  double kv_bytes_per_token; /* KV bytes of one token of one sequence, > 0 */
  int32_t num_layers;        /* L */
  int32_t attn_dim;          /* d: query heads x head size */
} tts_model_cost;

typedef struct {
  tts_model_cost verifier, generator;
  int64_t num_requests; /* N */
  int64_t verify_len;   /* S: verifier input length */
  int64_t decode_len;   /* S_dec: generated tokens per request */
  double mem_bytes;     /* M */
  double peak_flops;    /* P, FLOP/s */
  double peak_bw;       /* BW, bytes/s */
} tts_alloc_problem;

typedef struct {
  int64_t b_pre, b_dec;
  double t_tot, t_pre, t_dec; /* seconds */
} tts_alloc_result;

/* The modelled times of one choice (b_pre, b_dec >= 1; the memory budget is
 * not checked). */
tts_status tts_kv_alloc_time(const tts_alloc_problem* pr, int64_t b_pre, int64_t b_dec, tts_alloc_result* out);

/* The search; TTS_ERR_NOMEM when M holds no prefill and decode sequence. */
tts_status tts_kv_alloc_search(const tts_alloc_problem* pr, tts_alloc_result* out);

/* ---- Dynamic prefix-aware scheduling (Sec. 4.2) ----------------------------
 *
 * Orders the active reasoning paths (CoTs) of a search iteration so that
 * consecutive ones share long prefixes, and cuts the order into batches
 * that fit a KV budget. A CoT is a path of node ids from the root (a node
 * is a beam step; the ids of one CoT are distinct; CoT c is
 * cot_nodes[cot_offsets[c] .. cot_offsets[c + 1])). Order: CoT 0 first,
 * then repeatedly the remaining CoT with the longest common prefix with the
 * last one scheduled, ties to the earliest in the input (which keeps the
 * relative order of the parents' groups). Batches: from the front, the
 * longest run of consecutive CoTs whose trie (the union of their nodes,
 * each weighing node_weight[node], or 1 when node_weight is NULL) weighs at
 * most budget; a CoT heavier than the budget is a batch of its own.
 * Outputs (host, caller-allocated): order[num_cots]; batch_offsets
 * [num_batches + 1] (at most num_cots + 1) into order; score = the sum of
 * common-prefix lengths of consecutive CoTs; cost = sum over batches of
 * trie weight minus the weight shared with the next batch (the paper's
 * eviction cost). Host call. */
tts_status tts_prefix_schedule(int32_t num_cots, const int32_t* cot_offsets, const int32_t* cot_nodes,
                               int32_t num_nodes, const int64_t* node_weight, int64_t budget, int32_t* order,
                               int32_t* batch_offsets, int32_t* num_batches, int64_t* score, int64_t* cost);

/* Thread-local text of the last error ("" if none). */
const char* tts_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TTS_H_ */
