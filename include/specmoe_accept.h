/*
 * specmoe_accept.h -- greedy acceptance of draft tokens on MI355X (gfx950).
 *
 * After the target model has verified a chunk (specmoe_verify.h), the draft
 * tokens are checked against the target's own predictions (SpecMoEOff,
 * Section 2.3 "Speculative Decoding": the target model verifies the draft
 * tokens in one forward pass; Section 4.2 "Execution Workflow": the draft
 * model then updates its KV cache according to the verification result).
 * The paper does not spell out the rule; this library implements greedy
 * verification:
 *
 *   chunk b holds c_b tokens: token 0 is the last token already accepted,
 *   tokens 1..c_b-1 are drafts.  pred_i = argmax over the vocabulary of the
 *   logits at chunk position i (the lowest token id among equal values;
 *   +0 and -0 are equal).  a_b = the number of leading drafts with
 *   token[i+1] == pred_i for all i < a_b.  The next token is pred_{a_b}, and
 *   the first a_b + 1 chunk tokens become context: l_b <- l_b + a_b + 1.
 *   A sequence with c_b = 0 takes no step: a_b = 0, next token -1, l_b kept.
 *
 * Status codes are the SPECMOE_* values of specmoe_verify.h.  All functions
 * are plain C; pointers named "device" are HIP device pointers.
 */
#ifndef SPECMOE_ACCEPT_H
#define SPECMOE_ACCEPT_H

#include <stddef.h>
#include <stdint.h>

#include "specmoe_verify.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct specmoe_accept_desc {
  int32_t B;          /* sequences; 0 returns SPECMOE_OK at once                        */
  int32_t C_max;      /* chunk capacity: rows of logits / tokens per sequence, >= 1      */
  int32_t V;          /* vocabulary size, >= 1; V * element size must be a multiple of
                         16 bytes (rows are read in 16-byte vectors)                     */
  int32_t dtype;      /* specmoe_dtype of the logits (SPECMOE_F32 or SPECMOE_BF16)       */
  int32_t split;      /* vocabulary entries per work item; 0 = library default (8 KB
                         of logits); else a positive multiple of 512                     */
  int32_t flags;      /* reserved, must be 0                                             */
  void* workspace;          /* device; caller-allocated, >= workspace_bytes, counter
                               region zero before the first call (see below)            */
  size_t workspace_bytes;
} specmoe_accept_desc;

/*
 * specmoe_accept_greedy -- greedy acceptance of a batch of verified chunks.
 *
 * Arguments (device pointers, C-contiguous):
 *   logits       [B, C_max, V] dtype: the target's logits at every chunk
 *                position; rows i >= c_b are never read.  No NaN (a NaN
 *                logit gives an unspecified argmax, never an out-of-bounds
 *                access).  16-byte aligned.
 *   tokens       int32 [B, C_max]: chunk token ids (token 0 the last accepted
 *                token, then the drafts); entries i >= c_b are never read.
 *   ctx_lens     int32 [B]: l_b before the step.
 *   chunk_lens   int32 [B]: c_b; clamped into [0, C_max] before any access.
 *   argmax       int32 [B, C_max] out: pred_i for i < c_b, -1 beyond.
 *   accepted     int32 [B] out: a_b.
 *   next_token   int32 [B] out: pred_{a_b}, or -1 when c_b = 0.
 *   new_ctx_lens int32 [B] out: l_b + a_b + 1 (l_b when c_b = 0); may be the
 *                same buffer as ctx_lens (updated in place).
 *   stream       hipStream_t (NULL: the null stream).
 *
 * Work split: the valid rows' logits form a list of items of `split`
 * vocabulary entries; a persistent grid of waves takes contiguous ranges of
 * the list and stores one (max, first index) per row segment it covers; the
 * last wave of a sequence to finish (an arrival counter in the workspace)
 * combines the segments in vocabulary order, decides the acceptance and
 * writes the sequence's outputs.  Results do not depend on the split or on
 * timing.
 *
 * Workspace: a counter region (one int per sequence, left zero by every call
 * that completes) followed by the segment maxima.  Zero the counter region once
 * (specmoe_accept_workspace_init) before the first call; the workspace then
 * serves any number of calls with descriptors that need no more bytes.
 *
 * Ownership and errors as in specmoe_verify_attn: the caller owns every
 * buffer, nothing is allocated, nothing synchronises with the host, calls
 * that may overlap need distinct workspaces; all host checks run before any
 * HIP call and return SPECMOE_ERR_NULL_POINTER, SPECMOE_ERR_SHAPE (B < 0,
 * C_max < 1 or > 1024, B > 65536, V < 1, V * element size not a multiple of
 * 16, split not 0 or a positive multiple of 512, sizes past 32-bit index
 * arithmetic),
 * SPECMOE_ERR_DTYPE, SPECMOE_ERR_FLAGS, SPECMOE_ERR_ALIGN (logits or the
 * workspace not 16-byte aligned), SPECMOE_ERR_WORKSPACE or, from HIP,
 * SPECMOE_ERR_LAUNCH.
 */
int specmoe_accept_greedy(const void* logits, const int32_t* tokens, const int32_t* ctx_lens,
                          const int32_t* chunk_lens, int32_t* argmax, int32_t* accepted,
                          int32_t* next_token, int32_t* new_ctx_lens, void* stream,
                          const specmoe_accept_desc* desc);

/*
 * specmoe_accept_greedy_tree -- greedy acceptance of tree drafts.
 *
 * The chunk's tokens are the nodes of a draft tree in topological order
 * (Section 2.3: tree drafts are verified as a sequence plus a mask relating
 * them): node 0 is the last accepted token, the root; the parents come from
 * draft_mask, the root-path words of specmoe_verify_attn_tree (word i holds
 * the bits of i and its ancestors; a precondition).  Node i >= 1 is accepted
 * when its parent is and tokens[i] equals the prediction at the parent
 * (argmax of the parent's logits, ties to the lowest id).  The deepest
 * accepted node wins, the lowest index among equally deep ones; a_b is its
 * depth, the next token the prediction at it, new_ctx_lens = l_b + a_b + 1.
 *
 *   draft_mask   uint64 [B, C_max], device, 8-byte aligned; C_max <= 64
 *                (SPECMOE_ERR_MASK otherwise).
 *   path         uint64 [B] out, device, 8-byte aligned: the accepted path's
 *                node bits (the winning node's word; 0 when c_b = 0).
 * Every other argument, the workspace and the errors are those of
 * specmoe_accept_greedy.  Follow it with specmoe_compact_accepted_kv, with
 * the context lengths from before the step, to move the path's K/V rows
 * into place.
 */
int specmoe_accept_greedy_tree(const void* logits, const int32_t* tokens, const uint64_t* draft_mask,
                               const int32_t* ctx_lens, const int32_t* chunk_lens, int32_t* argmax,
                               int32_t* accepted, int32_t* next_token, int32_t* new_ctx_lens,
                               uint64_t* path, void* stream, const specmoe_accept_desc* desc);

/*
 * specmoe_compact_accepted_kv -- move an accepted tree path's K/V rows to
 * the rows right after the context (Section 4.2: the KV cache is updated
 * from the verification result).
 *
 * For every sequence b and KV head, the rows l_b + k of the set bits k of
 * path[b] (ascending) move to rows l_b + 0, 1, ...; all rows are read
 * before any is written.  Rows past S_max are skipped.
 *
 *   k_cache, v_cache  [B, Hkv, S_max, D] of desc's dtype, device, 16-byte
 *                aligned (a contiguous cache; desc->B, Hkv, D, S_max, dtype
 *                are used, the rest of desc is ignored).
 *   ctx_lens     int32 [B], device: l_b before the step (not the updated
 *                lengths).
 *   path         uint64 [B], device: as written by specmoe_accept_greedy_tree.
 * Status: SPECMOE_OK, SPECMOE_ERR_NULL_POINTER, SPECMOE_ERR_DTYPE,
 * SPECMOE_ERR_HEAD_DIM, SPECMOE_ERR_SHAPE, SPECMOE_ERR_ALIGN or
 * SPECMOE_ERR_LAUNCH.  Asynchronous on `stream`; allocates nothing.
 */
int specmoe_compact_accepted_kv(void* k_cache, void* v_cache, const int32_t* ctx_lens,
                                const uint64_t* path, void* stream, const specmoe_verify_desc* desc);

/* Bytes of workspace specmoe_accept_greedy needs for `desc`; 0 for an
 * invalid descriptor. */
size_t specmoe_accept_workspace_bytes(const specmoe_accept_desc* desc);

/* Zero the counter region of `workspace` with a small kernel on `stream`.
 * Status: SPECMOE_OK, a descriptor error, SPECMOE_ERR_NULL_POINTER,
 * SPECMOE_ERR_ALIGN, SPECMOE_ERR_WORKSPACE, or SPECMOE_ERR_LAUNCH. */
int specmoe_accept_workspace_init(void* workspace, size_t workspace_bytes, void* stream,
                                  const specmoe_accept_desc* desc);

#ifdef __cplusplus
}
#endif

#endif /* SPECMOE_ACCEPT_H */
