/*
 * evisel.h -- C ABI of libevisel.so, the MI355X (gfx950) sparse-prefill
 * evidence probe.
 *
 * The probe runs block-sparse causal attention over a packed batch of videos
 * laid out as X = [X_sys; X_vis; X_Q] (system prefix, N_v visual tokens per
 * anchor frame, query tokens), and in the same pass reduces the query rows'
 * softmax mass onto the anchor frames (the query-frame evidence cue). The
 * layout, the frame-aligned block partition, the always-visible system prefix
 * and the exact causal prefix of the current block follow the paper's
 * appendix "Detailed Sparse Prefilling"; the evidence follows "Evidence
 * Decomposition" (query-frame cue A_qf, timestamp-aligned E_qf, heads
 * averaged per layer).
 *
 * Conventions for every call:
 *  - Status codes, never exceptions. On failure nothing is launched and
 *    evisel_last_error() returns a message (thread-local, valid until the
 *    next failing call on the same thread).
 *  - "device" pointers are HIP device allocations on the current device;
 *    "host" pointers are ordinary host memory, read during the call only.
 *    Tensors are dense, row-major, 16-byte aligned.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Kernel work is asynchronous on it; results are valid once it syncs.
 *  - Tokens of all videos are packed: Q/O are [S, Hq, d], K/V [S, Hkv, d]
 *    with d contiguous. Query head h reads kv head h / (Hq / Hkv).
 */
#ifndef EVISEL_H
#define EVISEL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EVISEL_OK = 0,
  EVISEL_ERR_INVALID_ARG = 1, /* bad pointer, size or layout              */
  EVISEL_ERR_UNSUPPORTED = 2, /* valid but not implemented (d, B, N_v ...) */
  EVISEL_ERR_WORKSPACE = 3,   /* workspace missing or too small           */
  EVISEL_ERR_HIP = 4,         /* a HIP runtime call failed                */
  EVISEL_ERR_NOMEM = 5        /* host or device allocation failed         */
} evisel_status;

typedef enum { EVISEL_BF16 = 0, EVISEL_FP32 = 1 } evisel_dtype;

/* Packed batch of videos. Video n occupies n_sys[n] + n_frames[n] * N_v +
 * n_text[n] consecutive tokens, videos in order. Host memory, caller-owned,
 * read during evisel_build_block_mask only. n_sys may be NULL (all zero).
 * Requires n_seq >= 1, n_frames[n] >= 1, n_text[n] >= 1, n_sys[n] >= 0,
 * tokens_per_frame >= 1 and fewer than 2^31 tokens in total. */
typedef struct {
  int32_t n_seq;
  const int32_t* n_sys;
  const int32_t* n_frames;
  const int32_t* n_text;
  int32_t tokens_per_frame; /* N_v */
} evisel_layout;

/* Block-sparse rule (appendix: frame-aligned blocks of B tokens per region,
 * the last block of a region may be short). System-prefix tokens are visible
 * to every later token of their video; a token always sees the causal prefix
 * of its own block; videos never see each other.
 *
 * tau_p = 0: static rule. A visual query token in visual block b sees visual
 * blocks [0, sink_blocks), [b - window, b - 1] and its own block b up to
 * itself; window = -1 makes every preceding visual block visible (plain
 * causal attention). A query (text) token sees every visual block and the
 * query tokens up to itself.
 *
 * 0 < tau_p <= 1: the paper's adaptive top-p retention (appendix, mean-key,
 * affinity and probability equations). A video's selectable blocks are its
 * visual then query-token blocks, numbered 0, 1, ... in token order (the
 * "local" index); a token in local block b has the history H = local blocks
 * 0 .. b-1. Per query head and token, every history block j gets the
 * affinity g_j = q . kbar_j * softmax_scale, kbar_j the mean of block j's
 * keys (that head's kv head); p = softmax(g) over H; the token keeps the
 * smallest set of blocks, taken in decreasing p (equal p: lower index
 * first), whose total p reaches tau_p, and attends exactly to their tokens,
 * the system prefix and its own block's causal prefix. sink_blocks and
 * window are ignored. At most 2048 candidate key blocks per query block. */
typedef struct {
  int32_t block;       /* B >= 1; the attention kernel supports B = 64 */
  int32_t sink_blocks; /* >= 0 */
  int32_t window;      /* >= 0, or -1 for all-causal */
  float tau_p;         /* 0 (static rule) or (0, 1] (top-p retention) */
} evisel_mask_rule;

typedef struct evisel_mask evisel_mask; /* opaque, library-owned */

typedef struct {
  int64_t n_tokens;        /* S                                         */
  int64_t n_frames_total;  /* T = sum n_frames                          */
  int64_t n_text_rows;     /* sum n_text                                */
  int64_t n_blocks;        /* region blocks (query and key tiles)       */
  int64_t n_active_pairs;  /* active (query block, key block) pairs     */
  int64_t n_work_items;    /* attention work items (all heads)          */
  int64_t n_text_tiles;    /* query-token blocks                        */
  int64_t n_chunk_slots;   /* split query-token work items (all heads)  */
  int32_t hq, hkv, block, tokens_per_frame;
  int32_t hist_words;      /* W: 32-bit words of one row's history bits   */
  float tau_p;             /* the rule's tau_p                            */
  int64_t n_frame_pairs;   /* (frame, earlier frame) pairs the pattern can
                              connect: entries of the cross-frame cue      */
  int64_t n_paired_tiles;  /* key tiles of paired work items (below)      */
} evisel_mask_stats;

/* Builds the block partition, the compact list of active block pairs (CSR,
 * each row's key blocks in increasing order) and the attention work list
 * for Hq query heads and Hkv kv heads, then uploads them to the current
 * device. The upload is an asynchronous copy on `stream` from a pinned
 * host buffer the mask owns; the call does not wait for it. Compute calls
 * on the same stream are ordered after it; a caller that uses the mask on
 * another stream first synchronizes `stream` (or orders the other stream
 * after it). The device allocation and the pinned buffer are made here,
 * once per mask. *out is library-owned; release it with evisel_mask_free.
 * Errors: INVALID_ARG for a bad layout or rule or hq % hkv != 0, NOMEM,
 * HIP. */
evisel_status evisel_build_block_mask(const evisel_layout* layout,
                                      const evisel_mask_rule* rule,
                                      int32_t hq, int32_t hkv, void* stream,
                                      evisel_mask** out);

/* Same plan, host tables only (no device copy, no HIP call): for inspecting
 * the plan on a machine without a GPU. Such a mask is rejected by the
 * compute calls with INVALID_ARG. */
evisel_status evisel_build_block_mask_host(const evisel_layout* layout,
                                           const evisel_mask_rule* rule,
                                           int32_t hq, int32_t hkv,
                                           evisel_mask** out);

/* Frees host and device memory of a mask (NULL is ignored). It waits for
 * the mask's own upload copy; the caller must make sure no queued kernel
 * still reads the mask. */
void evisel_mask_free(evisel_mask* mask);

/* Reorders the attention work list: item i of the new launch order is item
 * perm[i] of the current one (perm: host [n_work_items], a permutation).
 * Every output of evisel_sparse_prefill has exactly one writer and every
 * reduction runs in a fixed order, so results do not depend on the launch
 * order; this call lets a caller check that (for example with the order
 * reversed). It waits for the mask's previous upload, then copies the new
 * work list asynchronously on `stream`. Errors: INVALID_ARG (host-only mask,
 * NULL perm, not a permutation), HIP. */
evisel_status evisel_mask_permute_work(evisel_mask* mask, const int32_t* perm,
                                       void* stream);

evisel_status evisel_mask_info(const evisel_mask* mask, evisel_mask_stats* out);

/* Copies the host plan into caller buffers (host memory; any may be NULL):
 * per block (n_blocks entries) its first token, length, region (0 system,
 * 1 visual, 2 query) and video; the CSR row_ptr (n_blocks + 1) and col
 * (n_active_pairs) over block indices. */
evisel_status evisel_mask_export(const evisel_mask* mask, int32_t* blk_start,
                                 int32_t* blk_len, int32_t* blk_region,
                                 int32_t* blk_video, int32_t* row_ptr,
                                 int32_t* col);

/* Copies the attention work list (n_work_items entries) in launch order:
 * query block (-1 for padding), first query head, number of query heads
 * (consecutive, sharing one kv head), first and one-past-last CSR position
 * of its key blocks, and the first head's split slot (-1 unless the item is
 * part of a split query-token row). Any pointer may be NULL.
 * With an odd number of query heads per kv head, the odd head of a kv
 * group is covered by paired items: one head over two
 * query blocks of the same video and region (qblock and qblock2 >= 0; for
 * split query-token rows, the same chunk of two consecutive query-token
 * blocks, with slots slot and slot2). A paired item's [kb_begin, kb_end)
 * indexes the paired-tile list of evisel_mask_export_paired instead of the
 * CSR. qblock2 and slot2 are -1 for every other item. */
evisel_status evisel_mask_export_work(const evisel_mask* mask, int32_t* qblock,
                                      int32_t* head, int32_t* nheads,
                                      int32_t* kb_begin, int32_t* kb_end,
                                      int32_t* slot, int32_t* qblock2,
                                      int32_t* slot2);

/* Copies the paired-tile list (n_paired_tiles entries): the key block and
 * its CSR position in the row of the paired item's first and second query
 * block (-1 where the key block is not active for that query block). The
 * tiles of one item are in increasing key-block order and are the union of
 * the two blocks' CSR runs. Any pointer may be NULL. */
evisel_status evisel_mask_export_paired(const evisel_mask* mask,
                                        int32_t* block, int32_t* pos_a,
                                        int32_t* pos_b);

/* Bytes of device workspace evisel_sparse_prefill (and, for a top-p mask,
 * evisel_select_blocks) needs for head dim d. */
size_t evisel_sparse_prefill_workspace(const evisel_mask* mask, int32_t d);

/* Extra workspace bytes, on top of evisel_sparse_prefill_workspace, that an
 * evisel_sparse_prefill call with frame_pairs or intra_frame needs. */
size_t evisel_cue_workspace(const evisel_mask* mask, int32_t d);

/* Copies the frame pairs of the cross-frame cue (n_frame_pairs entries) into
 * host buffers: query frame a and earlier key frame b (global frame ids, same
 * video). Pair i is entry i of evisel_sparse_prefill's frame_pairs. Either
 * pointer may be NULL. */
evisel_status evisel_mask_export_pairs(const evisel_mask* mask, int32_t* a,
                                       int32_t* b);

/* The paper's coarse query-frame evidence of one layer (appendix,
 * coarse-map equation; top-p masks only). For each query token i the tokens
 * of every retained history block j share the logit g_ij (the block
 * affinity of the retention step), the tokens of E_i (the video's system
 * prefix and the causal prefix of i's block) keep their exact logits
 * q_i . k_m * softmax_scale, and the row is normalised over both.
 *   evidence   device [Hq, T] fp32: per head and frame, the sum over the
 *              video's query tokens of that coarse probability on the
 *              frame's visual tokens (the coarse counterpart of
 *              evisel_sparse_prefill's evidence slice)
 * The call runs the retention itself (as evisel_select_blocks, into the
 * workspace) and then the coarse pass; no attention output is formed.
 * Errors: INVALID_ARG (static or host-only mask, NULL or misaligned
 * pointer), UNSUPPORTED (d, dtype, B), WORKSPACE, HIP. */
evisel_status evisel_coarse_evidence(const evisel_mask* mask, const void* q,
                                     const void* k, int32_t d,
                                     evisel_dtype dtype, float softmax_scale,
                                     float* evidence, void* workspace,
                                     size_t workspace_bytes, void* stream);

/* Top-p retention of one layer alone (appendix, mean-key, affinity and
 * probability equations and the smallest subset reaching tau_p; see
 * evisel_mask_rule). evisel_sparse_prefill runs the same kernels itself;
 * this call exposes their result.
 *   q, k, d, dtype, softmax_scale  as for evisel_sparse_prefill
 *   row_bits   device uint32 [Hq][n_blocks][W][64]: for query head h, query
 *              block qb and row r < 64 of the block, bit (j % 32) of word
 *              j / 32 is set when the row retains local history block j
 *              (W = hist_words of evisel_mask_info). Rows past the block's
 *              length, system-prefix blocks and blocks without history are
 *              all zero.
 *   block_bits device uint32 [Hq][n_blocks][W]: OR of the block's rows.
 *   workspace  as for evisel_sparse_prefill (only its mean-key region is
 *              used)
 * Probabilities, sums and the cut are computed in fp32; bf16 inputs use
 * bf16 MFMA with the block means split into two bf16 terms. Deterministic.
 * Errors: INVALID_ARG (host-only or static mask, NULL or misaligned
 * pointer), UNSUPPORTED (d, dtype, B), WORKSPACE, HIP. */
evisel_status evisel_select_blocks(const evisel_mask* mask, const void* q,
                                   const void* k, int32_t d,
                                   evisel_dtype dtype, float softmax_scale,
                                   uint32_t* row_bits, uint32_t* block_bits,
                                   void* workspace, size_t workspace_bytes,
                                   void* stream);

/* One layer of the probe (appendix sparse prefilling under the mask's rule;
 * evidence per Evidence Decomposition, query-frame cue). With a top-p mask
 * the call first runs the retention of evisel_select_blocks into the
 * workspace; key tiles that no row of a work item retained are skipped.
 *   q        device [S, Hq, d]   dtype
 *   k, v     device [S, Hkv, d]  dtype
 *   d        64 or 128; dtype EVISEL_BF16 or EVISEL_FP32
 *   softmax_scale  logit scale, normally 1/sqrt(d)
 *   out      device [S, Hq, d]   dtype: softmax(q k^T * scale) v over the
 *            visible keys (fp32 accumulation; bf16 output rounded to nearest
 *            even)
 *   lse      device [Hq, S] fp32, natural-log log-sum-exp of each row's
 *            scaled logits over its visible keys; may be NULL
 *   evidence device [n_layers, Hq, T] fp32; slice [layer] is overwritten
 *            with E[h, f] = sum over the query rows i of f's video of the
 *            softmax mass of row i on frame f's visual tokens (a raw sum
 *            over query rows, not a mean)
 *   text_mass device [n_layers, Hq, n_seq] fp32 or NULL; slice [layer] gets
 *            the same rows' mass on non-visual keys (system prefix and query
 *            tokens); per video sum_f E + text_mass = n_text
 *   frame_pairs device [n_layers, n_frame_pairs] fp32 or NULL: the
 *            cross-frame cue (Evidence Decomposition, A_ff). Entry i of
 *            slice [layer] is, for pair (a, b) of evisel_mask_export_pairs,
 *            the mean over heads and over frame a's N_v rows of the row's
 *            total probability on frame b's visual tokens. Pairs outside
 *            the list are 0.
 *   intra_frame device [n_layers, T, N_v, N_v] fp32 or NULL: the intra-frame
 *            cue (A_if; flattened per timestamp it is E_if). Slice [layer]
 *            [t][i][m] is the head mean of the probability of frame t's
 *            token i on its token m (0 for m > i).
 *   workspace device, >= evisel_sparse_prefill_workspace(mask, d) bytes,
 *            plus evisel_cue_workspace(mask, d) when frame_pairs or
 *            intra_frame is given
 * Requires B = 64, N_v dividing 64 with N_v >= 8 (when any video has
 * query rows reducing onto frames), 0 <= layer < n_layers.
 * Errors: INVALID_ARG (NULL buffer, host-only mask, layer out of range),
 * UNSUPPORTED (d, dtype, B or N_v), WORKSPACE, HIP (launch failure). */
evisel_status evisel_sparse_prefill(const evisel_mask* mask, int32_t layer,
                                    int32_t n_layers, const void* q,
                                    const void* k, const void* v, int32_t d,
                                    evisel_dtype dtype, float softmax_scale,
                                    void* out, float* lse, float* evidence,
                                    float* text_mass, float* frame_pairs,
                                    float* intra_frame, void* workspace,
                                    size_t workspace_bytes, void* stream);

/* Bytes of the static workspace of evisel_sparse_prefill_noalloc, per GPU. */
#define EVISEL_NOALLOC_WORKSPACE_BYTES ((size_t)64 << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * evisel_sparse_prefill with the same arguments and results, minus
 * workspace and workspace_bytes. The workspace is a device array inside the
 * library, EVISEL_NOALLOC_WORKSPACE_BYTES on every GPU the library is loaded
 * on, held until the process ends. The call allocates nothing and clears
 * nothing: no kernel of a call reads workspace bytes that the same call has
 * not written, so the array keeping the previous call's contents does not
 * matter. Every call on one GPU shares that GPU's array: calls that overlap
 * on one GPU (two streams, or two host threads) race, and the caller must
 * order them (e.g. one stream). The array's device address is looked up on
 * the first call on each GPU.
 * Errors: those of evisel_sparse_prefill; WORKSPACE when the mask (with the
 * frame-cue workspace, when frame_pairs or intra_frame is given) needs more
 * than EVISEL_NOALLOC_WORKSPACE_BYTES; UNSUPPORTED for a device ordinal
 * above 63. */
evisel_status evisel_sparse_prefill_noalloc(
    const evisel_mask* mask, int32_t layer, int32_t n_layers, const void* q,
    const void* k, const void* v, int32_t d, evisel_dtype dtype,
    float softmax_scale, void* out, float* lse, float* evidence,
    float* text_mass, float* frame_pairs, float* intra_frame, void* stream);

/* Aggregates evidence [n_layers, Hq, T] (Evidence Decomposition: mean over
 * heads per layer, then the timestamp-aligned query-frame score):
 *   e_qf_layer device [n_layers, T] or NULL:
 *              sum_h E[l, h, t] / (Hq * n_text(video of t))
 *   e_qf       device [T]: mean over layers of e_qf_layer
 *   k_per_seq  device [n_seq] int32, or NULL (no top-k); each value is
 *              clamped to [0, n_frames[n]]
 *   topk_idx   device [sum of clamped k] int32: per video, in video order,
 *              the k local frame indices with the largest e_qf, ordered by
 *              (e_qf descending, index ascending); NaN ranks as -inf
 *   frame_pairs device [n_layers, n_frame_pairs] from evisel_sparse_prefill,
 *              or NULL
 *   e_ff       device [n_layers, T] or NULL (needs frame_pairs): the
 *              timestamp-aligned cross-frame evidence. For frame t at local
 *              index t' of a video with F frames: the mean over its t'
 *              earlier frames b of A_ff[t, b] and the mean over its F-1-t'
 *              later frames a of A_ff[a, t], averaged over the sides that
 *              exist (0 for a one-frame video)
 * Errors: INVALID_ARG, UNSUPPORTED (a video with more than 65536 frames
 * when top-k is requested), HIP. */
evisel_status evisel_frame_evidence(const evisel_mask* mask,
                                    const float* evidence, int32_t n_layers,
                                    float* e_qf_layer, float* e_qf,
                                    const int32_t* k_per_seq,
                                    int32_t* topk_idx,
                                    const float* frame_pairs, float* e_ff,
                                    void* stream);

/* Kernel timing, a tracing aid. evisel_profile_begin creates 5 * capacity
 * HIP events on the current device. The evisel_sparse_prefill calls that
 * follow are counted from 0; calls 0, stride, 2 * stride, ... are timed, up
 * to `capacity` timed calls, and the others record nothing. With
 * all_kernels != 0 a timed call records events on its stream before the
 * top-p retention (empty for a static mask), before the attention kernel,
 * after it, after the kernel that merges the split query rows and reduces
 * the evidence, and after the frame cues (empty when none is requested).
 * With all_kernels == 0 it records only the two events around the attention
 * kernel, so that the other kernels run back to back. Each event is a
 * dependency packet that leaves the GPU idle for several microseconds,
 * hence the stride. evisel_profile_end waits for those events, writes the
 * summed milliseconds of the four spans into ms[0..3] (retention,
 * attention, combine and evidence, cues; spans that were not recorded are
 * 0) and the number of timed calls (either pointer may be NULL) and
 * destroys the events. One session at a time per process; not thread-safe.
 * Errors: INVALID_ARG (capacity < 1, stride < 1, a session already open or
 * none open), NOMEM, HIP. */
evisel_status evisel_profile_begin(int32_t capacity, int32_t all_kernels,
                                   int32_t stride);
evisel_status evisel_profile_end(double* ms, int64_t* n_calls);

/* Message of the last failing call on this thread ("" if none). */
const char* evisel_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* EVISEL_H */
