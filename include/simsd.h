/*
 * simsd.h -- C ABI of the SimSD verification step on AMD Instinct MI355X (gfx950).
 *
 * SimSD ("Simple Speculative Decoding in Diffusion Language Models") verifies
 * gamma drafted tokens of a block-diffusion LM in ONE target forward pass.
 * Each new sequence position appears twice: a block slot (the mask section,
 * where the target predicts) and, for drafted positions, a reference slot (the
 * data section, holding the drafted token).  A token-level temporal mask (Sec.
 * 3.1, eq. 1) lets the verification slot of draft r see the prompt and drafts
 * 1..r-1 only, so all gamma target distributions come out of one pass (Sec.
 * 3.2).  Acceptance keeps the longest prefix of drafts that pass eq. 2.
 *
 * This library computes the two data-parallel steps of that pass:
 *   simsd_verify_attention  attention of every new slot over [cached prefix |
 *                           new slots] under the temporal mask (generated on the
 *                           fly, never stored), GQA-packed, split over the prefix;
 *   simsd_verify_accept     vocabulary scan of the verification rows (argmax with
 *                           lowest-index ties, confidence, draft probability) and
 *                           the accepted-prefix length, i.e. eq. 2 at temperature 0;
 *   simsd_verify_accept_sampled  eq. 2 at temperature T: acceptance with
 *                           probability min(1, p_theta/p_phi) and the residual
 *                           draw at the first rejection.
 *
 * Conventions shared by both calls
 * --------------------------------
 *  - Sizes are element counts.  All tensors are row-major and densely packed
 *    unless a stride is given.  "b" = batch index.
 *  - New slots of a sequence: n_new = B + L, where B = block_size and
 *    L = max_ref.  Slot k < B is block slot k (the mask section).  Slot B + r
 *    is reference slot r, holding draft r+1 (the data section, Sec. 3.2).
 *  - step_map[b, k] (int32, one per block slot) extends the paper's step map
 *    (Sec. 3.1):
 *        1..gamma_b  block slot k is verified at draft step r (it is o_r);
 *        0           position committed before this step (visible to every
 *                    non-padded row, like the prompt);
 *        > gamma_b   position not drafted in this step (a mask placeholder at
 *                    every step);
 *        < 0         padding (its row outputs nothing, its column is unseen).
 *    num_ref[b] = gamma_b <= L; reference slots r >= gamma_b are padding.
 *    Each value 1..gamma_b must occur exactly once per sequence; the kernels
 *    do not check this (simsd_validate_step_map does, on the host).
 *  - Every pointer argument of the two compute calls is device memory owned by
 *    the caller.  The library allocates nothing, frees nothing and never
 *    synchronises: both calls only enqueue work on `stream` (a hipStream_t
 *    passed as void*; NULL = the default stream) and return.
 *  - Errors: the host checks shapes, dtypes, null pointers, 16-byte alignment
 *    and workspace size before anything is enqueued and returns a status other
 *    than SIMSD_OK, with a message in simsd_last_error() (thread-local).  A
 *    failed launch returns SIMSD_ERR_HIP.  No C++ exception crosses the ABI.
 *    Data-dependent preconditions are not checked on the device and violating
 *    them is undefined: step maps as above, 0 <= prefix_lens[b] <=
 *    max_prefix_len, block_table ids inside the page pool, finite inputs.
 *  - Workspace: caller-owned device memory of at least the size the matching
 *    *_workspace_size() call returns (it may be 0, and then the pointer may
 *    be NULL).  It holds per-chunk partial results between the kernels of one
 *    call; its contents need no initialisation and are meaningless afterwards.
 *    Two calls in flight at the same time need two workspaces.
 *  - Grid sizes follow the compute-unit count of the device a call's stream
 *    belongs to (queried once per device through the HIP device attributes
 *    and cached; a compute-partitioned MI355X reports its partition's units).
 *    The *_workspace_size() calls size for the current device (for an
 *    MI355X's 256 units when no device is visible); a call on a device with
 *    more units may need more and then returns SIMSD_ERR_WORKSPACE.  If the
 *    device query fails, argument errors are still reported first, then
 *    SIMSD_ERR_HIP.
 */
#ifndef SIMSD_H
#define SIMSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SIMSD_VERSION 100 /* 1.0.0 */

typedef enum {
  SIMSD_OK = 0,
  SIMSD_ERR_NULL_POINTER = 1,     /* a required pointer is NULL                       */
  SIMSD_ERR_BAD_SHAPE = 2,        /* inconsistent or out-of-range sizes/strides       */
  SIMSD_ERR_UNSUPPORTED = 3,      /* valid but not implemented (dtype, head_dim)      */
  SIMSD_ERR_ALIGNMENT = 4,        /* a pointer or stride is not 16-byte aligned       */
  SIMSD_ERR_WORKSPACE = 5,        /* workspace missing or smaller than required       */
  SIMSD_ERR_INVALID_STEP_MAP = 6, /* simsd_validate_step_map found a bad step map     */
  SIMSD_ERR_HIP = 7               /* the HIP runtime reported an error (device query
                                     or launch)                                       */
} simsd_status;

typedef enum {
  SIMSD_F32 = 0,  /* IEEE binary32                                      */
  SIMSD_BF16 = 1  /* bfloat16 (upper 16 bits of a binary32), RNE output  */
} simsd_dtype;

/* ------------------------------------------------------------------------ */
/* Verification attention                                                     */
/* ------------------------------------------------------------------------ */

/*
 * Shape of one verification-attention call.
 *
 * Query head h uses KV head h / (num_q_heads / num_kv_heads).  Scores are
 * scale * (q . k); scale == 0 selects 1/sqrt(head_dim).
 *
 * Cache layout.  page_size == 0: contiguous, element (b, t, h, i) of the
 * prefix at  cache[b*cache_stride_seq + t*cache_stride_token +
 * h*cache_stride_head + i]  for t < prefix_lens[b] <= max_prefix_len.
 * page_size > 0: paged, token t of sequence b lives in page
 * p = block_table[b*max_pages_per_seq + t/page_size] at row t % page_size:
 * cache[p*cache_stride_seq + (t%page_size)*cache_stride_token +
 * h*cache_stride_head + i]  (cache_stride_seq is then the page stride).
 * The same layout and strides apply to k_cache and v_cache.  Strides are in
 * elements, non-negative, at most 2^48, and must be multiples of 16 bytes.
 * The last index (head_dim) is contiguous.
 */
typedef struct {
  int32_t batch;              /* sequences, >= 1                                  */
  int32_t num_q_heads;        /* Hq >= 1                                          */
  int32_t num_kv_heads;       /* Hkv >= 1, Hq % Hkv == 0, Hq / Hkv <= 16          */
  int32_t head_dim;           /* 64 or 128                                        */
  int32_t block_size;         /* B >= 1                                           */
  int32_t max_ref;            /* L, 0 <= L <= B, B + L <= 64                      */
  int32_t max_prefix_len;     /* upper bound of prefix_lens[], >= 0               */
  int32_t page_size;          /* 0 = contiguous cache; else tokens per page       */
  int32_t max_pages_per_seq;  /* paged: block_table row length,
                                 >= ceil(max_prefix_len / page_size)              */
  int32_t kv_chunk;           /* prefix keys per work-group (multiple of 64);
                                 0 to let the library choose; -1 for the stream
                                 decomposition (equal tile ranges per resident
                                 work-group; bf16, Hq/Hkv*(B+L) <= 128 and
                                 batch <= 256 only, else SIMSD_ERR_UNSUPPORTED) */
  int64_t cache_stride_seq;   /* elements between sequences (contiguous) / pages  */
  int64_t cache_stride_token; /* elements between consecutive tokens              */
  int64_t cache_stride_head;  /* elements between consecutive KV heads            */
  float scale;                /* softmax scale; 0 = 1/sqrt(head_dim)              */
  simsd_dtype dtype;          /* of q, k_new, v_new, k_cache, v_cache and out     */
  float rope_theta;           /* 0: q and k_new arrive rotated.  > 0: they arrive
                                 unrotated and the kernels apply the rotary
                                 embedding with this base at the RoPE-copy
                                 positions (see simsd_verify_attention)          */
} simsd_attn_desc;

/* Bytes of workspace simsd_verify_attention needs for `desc` (host only; 0 for
 * an invalid descriptor, whose error simsd_verify_attention reports). */
size_t simsd_verify_attention_workspace_size(const simsd_attn_desc* desc);

/*
 * Attention of every new slot over its visible keys (Sec. 3.2, "Target Model
 * Verification"; mask: Sec. 3.1, eq. 1; the prompt is visible to every
 * non-padded response row, padding rows/columns are removed).
 *
 *   q       [batch, B+L, Hq,  head_dim]  queries of the new slots (after RoPE,
 *                                        or before it when rope_theta > 0)
 *   k_new   [batch, B+L, Hkv, head_dim]  keys of the new slots (likewise)
 *   v_new   [batch, B+L, Hkv, head_dim]  values of the new slots
 *   k_cache, v_cache                     cached prefix, layout above
 *   block_table [batch, max_pages_per_seq] int32, or NULL if page_size == 0
 *   prefix_lens [batch] int32            cached prefix length of each sequence
 *   step_map    [batch, B] int32         see the conventions above
 *   num_ref     [batch] int32            gamma_b
 *   out     [batch, B+L, Hq, head_dim]   softmax(scale q K^T) V over the visible
 *                                        keys, in `dtype` (bf16 rounded to
 *                                        nearest even); padding rows are 0
 *   lse     [batch, Hq, B+L] float32     natural-log log-sum-exp of the scaled
 *                                        scores of each row (-inf for padding
 *                                        rows), or NULL
 *   workspace, workspace_bytes           see the conventions above
 *   stream                               hipStream_t
 *
 * RoPE copy (Sec. 3.1, Sec. 3.2), when rope_theta > 0: dims i and i + d/2 of
 * each new slot's query and key are rotated by pos * rope_theta^(-2i/d), in
 * fp32, before the scores (the new keys are rounded back to the input dtype).
 * Block slot k sits at pos = prefix_lens[b] + k; reference slot r (draft r+1)
 * shares the index of its verification slot, prefix_lens[b] + k_{r+1}, where
 * step_map[b, k_{r+1}] = r + 1; padding reference slots take prefix_lens[b].
 * The cached prefix keys must already be rotated at indices 0..prefix_len-1.
 * rope_theta must be finite and >= 0 (SIMSD_ERR_BAD_SHAPE otherwise).
 */
simsd_status simsd_verify_attention(const simsd_attn_desc* desc, const void* q,
                                    const void* k_new, const void* v_new,
                                    const void* k_cache, const void* v_cache,
                                    const int32_t* block_table, const int32_t* prefix_lens,
                                    const int32_t* step_map, const int32_t* num_ref,
                                    void* out, float* lse, void* workspace,
                                    size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Vocabulary scan and acceptance                                            */
/* ------------------------------------------------------------------------ */

typedef struct {
  int32_t batch;             /* sequences, >= 1                                    */
  int32_t block_size;        /* B, 1 <= B <= 64                                    */
  int32_t max_ref;           /* L, 0 <= L <= B                                     */
  int32_t vocab;             /* V >= 1                                             */
  int32_t chunks_per_row;    /* work-groups per logits row, or 0 = library's choice */
  simsd_dtype logits_dtype;  /* of logits                                          */
} simsd_accept_desc;

size_t simsd_verify_accept_workspace_size(const simsd_accept_desc* desc);

/*
 * Greedy verification (eq. 2 at temperature 0, Sec. 3.2): draft r is accepted
 * while the target's argmax at its verification slot equals it; the longest
 * accepted prefix is kept.
 *
 *   logits      [batch, B, V]   row k = target logits at block slot k.  Only
 *                               rows with step_map >= 1 are read.
 *   draft_ids   [batch, L] int32  draft r at index r-1 (entries >= gamma_b unused)
 *   step_map, num_ref           as for simsd_verify_attention
 *   target_ids  [batch, B] int32   smallest index of the row maximum (stored
 *                                  values compared exactly, -0 == +0), or -1
 *                                  for rows that are not scanned
 *   confidence  [batch, B] float32 largest softmax probability of the row
 *                                  (0 for rows not scanned), or NULL
 *   draft_prob  [batch, L] float32 target softmax probability of draft r at
 *                                  its verification row; 0 for an id outside
 *                                  [0, V) and for r >= gamma_b; or NULL
 *   accept_len  [batch] int32      largest a <= gamma_b such that drafts
 *                                  1..a all equal their rows' target_ids.  A
 *                                  draft id outside [0, V) is a rejection.
 *                                  On rejection the correction token is
 *                                  target_ids at the row of draft a+1.
 */
simsd_status simsd_verify_accept(const simsd_accept_desc* desc, const void* logits,
                                 const int32_t* draft_ids, const int32_t* step_map,
                                 const int32_t* num_ref, int32_t* target_ids,
                                 float* confidence, float* draft_prob, int32_t* accept_len,
                                 void* workspace, size_t workspace_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the greedy
 * verification of simsd_verify_accept with no workspace argument.  The scan
 * partials go to a fixed device array of SIMSD_NOALLOC_SCRATCH_BYTES inside the
 * library; each GPU the library runs on holds its own copy of it until the
 * process ends.
 *
 *   desc, logits, draft_ids, step_map, num_ref, target_ids, confidence,
 *   draft_prob, accept_len, stream     exactly as for simsd_verify_accept,
 *                                      and the outputs are the same bits
 *
 * Nothing is allocated, freed or synchronised by the call; its first call on a
 * device looks up that device's copy of the array (making the device current
 * for the lookup and restoring the previous one).  Shapes whose partials need
 * more than SIMSD_NOALLOC_SCRATCH_BYTES (16 bytes per scanned row and
 * vocabulary chunk, the size simsd_verify_accept_workspace_size reports)
 * return SIMSD_ERR_WORKSPACE with nothing enqueued: use simsd_verify_accept
 * with a workspace for those.  All calls on one GPU share its array, which
 * keeps the last call's contents (every entry is written before it is read, so
 * nothing needs clearing): calls that overlap on one GPU, on any streams, race
 * and must be serialised by the caller.  Other errors as simsd_verify_accept;
 * SIMSD_ERR_HIP also if the array's device address cannot be obtained.
 */
#define SIMSD_NOALLOC_SCRATCH_BYTES ((size_t)4 << 20) /* 4 MiB per device */
simsd_status simsd_verify_accept_noalloc(const simsd_accept_desc* desc, const void* logits,
                                         const int32_t* draft_ids, const int32_t* step_map,
                                         const int32_t* num_ref, int32_t* target_ids,
                                         float* confidence, float* draft_prob,
                                         int32_t* accept_len, void* stream);

/*
 * Stochastic verification (eq. 2 at temperature T > 0, Sec. 3.2; the paper's
 * experiments use T = 1, Sec. 4.1): the rule the greedy call is the T -> 0
 * limit of.  With p_theta(r) = softmax(logits[b, k_r] / T) at the
 * verification row k_r of draft r and p_phi(r) = softmax(draft_logits[b, r-1]
 * / T), draft r is accepted iff u_r * p_phi(r)(D_r) < p_theta(r)(D_r), which
 * for u_r ~ U[0, 1) happens with probability min(1, p_theta / p_phi).  The
 * longest accepted prefix is kept; at the first rejected draft a+1 the target's
 * token is drawn from the residual max(0, p_theta(a+1) - p_phi(a+1)) by
 * inverse CDF in vocabulary order: the smallest x whose running weight exceeds
 * w * (total weight), w = uniforms[b, L].  If the residual is zero everywhere
 * the draw uses p_theta(a+1).  The random numbers are the caller's.
 *
 *   temperature  T, finite and > 0 (else SIMSD_ERR_BAD_SHAPE)
 *   logits       [batch, B, V]  target logits; rows of steps 1..gamma_b are read
 *   draft_logits [batch, L, V]  row r-1 = the drafter's logits when it proposed
 *                               draft r (same dtype as logits, 16-byte aligned);
 *                               rows r-1 < gamma_b are read.  NULL only if L = 0
 *   draft_ids    [batch, L] int32
 *   step_map, num_ref           as for simsd_verify_attention
 *   uniforms     [batch, L + 1] float32 in [0, 1): u_1..u_L, then w
 *   p_target     [batch, L] float32  p_theta(r)(D_r), 0 for an id outside
 *                                    [0, V) and for r > gamma_b; or NULL
 *   p_draft      [batch, L] float32  p_phi(r)(D_r), likewise; or NULL
 *   accept_len   [batch] int32       accepted drafts, 0..gamma_b.  A draft id
 *                                    outside [0, V) is a rejection.
 *   correction   [batch] int32       token drawn at the first rejection, or -1
 *                                    when every draft was accepted
 * Probabilities and running sums are float32: the draw can differ from an
 * exact one only where w * total falls within rounding of a boundary.
 * The workspace must hold simsd_verify_accept_sampled_workspace_size() bytes.
 */
size_t simsd_verify_accept_sampled_workspace_size(const simsd_accept_desc* desc);
simsd_status simsd_verify_accept_sampled(const simsd_accept_desc* desc, float temperature,
                                         const void* logits, const void* draft_logits,
                                         const int32_t* draft_ids, const int32_t* step_map,
                                         const int32_t* num_ref, const float* uniforms,
                                         float* p_target, float* p_draft, int32_t* accept_len,
                                         int32_t* correction, void* workspace,
                                         size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* LM head fused with the scan                                                */
/* ------------------------------------------------------------------------ */

typedef struct {
  int32_t batch;             /* sequences, >= 1                                    */
  int32_t block_size;        /* B, 1 <= B <= 64                                    */
  int32_t max_ref;           /* L, 0 <= L <= B                                     */
  int32_t vocab;             /* V >= 1                                             */
  int32_t hidden;            /* H, a positive multiple of 64                       */
  simsd_dtype dtype;         /* of hidden and weight: SIMSD_BF16 only              */
} simsd_lmhead_desc;

size_t simsd_verify_accept_lmhead_workspace_size(const simsd_lmhead_desc* desc);

/*
 * Greedy verification as simsd_verify_accept, with the logits computed on
 * the fly from the verification rows' final hidden states and the LM-head
 * weight (the target model's prediction at each verification slot, Sec. 3.2):
 * logits[b, k, v] = hidden[b, k, :] . weight[v, :], accumulated in fp32 from
 * bf16 products, never stored.  Outputs and their meaning are those of
 * simsd_verify_accept (ties between exactly equal fp32 logits go to the lowest
 * index).
 *
 *   hidden  [batch, B, H] bf16, 16-byte aligned; row k = block slot k
 *   weight  [V, H] bf16, 16-byte aligned (a Linear layer's [out, in] layout)
 *   draft_ids, step_map, num_ref, target_ids, confidence, draft_prob,
 *   accept_len, workspace, workspace_bytes, stream   as for simsd_verify_accept
 *   (draft_ids may be NULL when max_ref == 0; confidence and draft_prob may be
 *   NULL)
 * The workspace must hold simsd_verify_accept_lmhead_workspace_size() bytes
 * (0 for an invalid descriptor), 16-byte aligned, no initialisation needed; it
 * is fully rewritten by each call, so calls on one stream may share it.  All
 * buffers belong to the caller; the library allocates nothing and does not
 * synchronise.  Three kernels are enqueued on the stream.  The fp32
 * accumulation order is fixed for a given shape, so repeated calls give the
 * same bits.
 * Errors (nothing is enqueued): SIMSD_ERR_NULL_POINTER, SIMSD_ERR_BAD_SHAPE
 * (descriptor out of range, H not a multiple of 64), SIMSD_ERR_UNSUPPORTED
 * (dtype other than SIMSD_BF16), SIMSD_ERR_ALIGNMENT (hidden, weight or
 * workspace), SIMSD_ERR_WORKSPACE; SIMSD_ERR_HIP if a launch fails.
 */
simsd_status simsd_verify_accept_lmhead(const simsd_lmhead_desc* desc, const void* hidden,
                                        const void* weight, const int32_t* draft_ids,
                                        const int32_t* step_map, const int32_t* num_ref,
                                        int32_t* target_ids, float* confidence, float* draft_prob,
                                        int32_t* accept_len, void* workspace,
                                        size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Host-only helpers (no GPU needed)                                          */
/* ------------------------------------------------------------------------ */

/* Checks host copies of step_map [batch, B] and num_ref [batch]: 0 <= gamma_b
 * <= L and every value 1..gamma_b exactly once per sequence.  Returns SIMSD_OK
 * or SIMSD_ERR_INVALID_STEP_MAP (SIMSD_ERR_NULL_POINTER / _BAD_SHAPE for bad
 * arguments: batch >= 1, 1 <= B <= 64, 0 <= L <= B), with the first offending
 * sequence in simsd_last_error(). */
simsd_status simsd_validate_step_map(const int32_t* step_map_host, const int32_t* num_ref_host,
                                     int32_t batch, int32_t block_size, int32_t max_ref);

const char* simsd_status_string(simsd_status status);
const char* simsd_last_error(void); /* message of this thread's last failed call */
int simsd_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SIMSD_H */
