/*
 * specmoe_verify.h -- chunked verification attention on MI355X (gfx950).
 *
 * The operation is the chunked-attention operator of speculative-decoding
 * verification (SpecMoEOff, Section 5.1 "Chunked Attention in Target Model
 * Verification"): for every sequence b, the n = c_b draft tokens of its chunk
 * attend to the l = l_b cached tokens of its KV cache plus the chunk's own
 * tokens.  With Q in R^{n x d}, K, V in R^{(l+n) x d} and the additive mask
 * M in {-inf, 0}^{n x (l+n)} (draft token i sees every cached token and draft
 * tokens 0..i, i.e. key positions j <= l + i):
 *
 *     out = softmax(scale * Q K^T + M) V,   lse = log sum_j exp(scale q.k_j + M_ij)
 *
 * per query head, with grouped-query attention: g = Hq / Hkv query heads share
 * one KV head and query head h reads KV head h / g (the paper's group factor g,
 * Section 3.1 "Model").  The KV cache is the paper's 4-D [b, h, s, d] layout
 * (Section 5.2, "CPU/GPU separation for Draft Model Execution").
 *
 * Entry points: specmoe_verify_attn (chain drafts, the mask above),
 * specmoe_verify_attn_tree (tree drafts: the draft part of the mask given as
 * one bit word per draft token), specmoe_verify_attn_paged (either, over a
 * paged KV cache).  q, k and v may be float32, bfloat16 or float16 (the
 * paper's KV precision, Section 3.3).  The acceptance step that follows
 * verification is in specmoe_accept.h.
 *
 * All functions are plain C; every pointer named "device" is a HIP device
 * pointer, every other pointer is a host pointer.
 */
#ifndef SPECMOE_VERIFY_H
#define SPECMOE_VERIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of q, k_cache and v_cache.  out and lse are always float32.
 * FP16 is the KV precision the paper assumes (Section 3.3, Section 6.1). */
typedef enum {
  SPECMOE_F32 = 0,
  SPECMOE_BF16 = 1,
  SPECMOE_F16 = 2
} specmoe_dtype;

/* Status codes returned by the entry points (0 = success). */
enum {
  SPECMOE_OK = 0,
  SPECMOE_ERR_NULL_POINTER = -1,  /* a required pointer (or the descriptor) is NULL   */
  SPECMOE_ERR_SHAPE = -2,         /* B < 0, Hq/Hkv <= 0, C_max < 1, S_max < C_max, or
                                     sizes too large for the index arithmetic         */
  SPECMOE_ERR_GQA = -3,           /* Hq is not a multiple of Hkv                      */
  SPECMOE_ERR_HEAD_DIM = -4,      /* D is not 64 or 128                               */
  SPECMOE_ERR_DTYPE = -5,         /* dtype is not a specmoe_dtype value               */
  SPECMOE_ERR_ROWS = -6,          /* C_max * (Hq / Hkv) > 128 query rows per KV head  */
  SPECMOE_ERR_GRID = -7,          /* grid_blocks is negative, larger than 2048, or so
                                     large that partial results would pass 2 GB       */
  SPECMOE_ERR_WORKSPACE = -8,     /* workspace smaller than the size query returns    */
  SPECMOE_ERR_ALIGN = -9,         /* q, k_cache, v_cache, out or workspace is not
                                     16-byte aligned, or draft_mask not 8-byte aligned */
  SPECMOE_ERR_SCALE = -10,        /* scale is not finite and positive                 */
  SPECMOE_ERR_LAUNCH = -11,       /* HIP reported an error for a kernel launch        */
  SPECMOE_ERR_FLAGS = -12,        /* flags holds a bit other than SPECMOE_FLAG_NO_WAIT */
  SPECMOE_ERR_MASK = -13,         /* a draft mask with C_max > 64 (one 64-bit word per
                                     draft token covers at most 64 draft tokens)      */
  SPECMOE_ERR_PAGES = -14,        /* paged cache: page_size not a power of two in
                                     [8, 65536], pages_per_seq or num_pages < 1, or
                                     S_max != page_size * pages_per_seq               */
  SPECMOE_ERR_HANDOFF = -15       /* (specmoe_verify_attn_status) a kernel's wait for
                                     another wave of its workgroup gave up: the
                                     results of that call are unspecified            */
};

/* desc->flags bits. */
enum {
  /* Diagnostics only: every in-kernel wait for another wave gives up after a
   * single check instead of polling for about 0.1 s.  The kernels still end
   * normally and stay inside every buffer, but the results are unspecified
   * and the workspace's status word records the give-up (see
   * specmoe_verify_attn_status).  It exists to exercise that reporting. */
  SPECMOE_FLAG_NO_WAIT = 1
};

/* Problem description.  Sizes are in elements unless stated otherwise. */
typedef struct specmoe_verify_desc {
  int32_t B;          /* sequences in the batch; 0 returns SPECMOE_OK at once, without
                         looking at any data pointer                              */
  int32_t Hq;         /* query heads                                                */
  int32_t Hkv;        /* KV heads; Hq % Hkv == 0, g = Hq / Hkv                      */
  int32_t D;          /* head dimension: 64 or 128                                  */
  int32_t C_max;      /* draft-token capacity per sequence (rows of q/out/lse)      */
  int32_t S_max;      /* token capacity of the KV cache per (sequence, KV head)     */
  int32_t dtype;      /* specmoe_dtype of q, k_cache, v_cache                       */
  int32_t grid_blocks;  /* persistent workgroups that share the key tiles; 0 = the
                           library default (256: one per CU of an MI355X)          */
  int32_t flags;        /* 0, or SPECMOE_FLAG_NO_WAIT (diagnostics)                */
  void* workspace;          /* device; caller-allocated scratch, >= workspace_bytes,
                               whose zeroed region is zero (see below)              */
  size_t workspace_bytes;   /* size of workspace in bytes                           */
} specmoe_verify_desc;

/*
 * specmoe_verify_attn -- chunked verification attention (Section 5.1).
 *
 * Work split: the keys of every (sequence, KV head) are cut into tiles, and
 * the tiles of all of them are divided into at most `grid_blocks` contiguous
 * ranges of equal cost, one per persistent workgroup; a tile's cost grows
 * with the query rows (c_b * Hq / Hkv) that compute on it, so with equal
 * chunk lengths every range holds the same number of tiles (give or take
 * one).  A (sequence, KV head) whose tiles
 * span several ranges is computed in pieces that are merged with log-sum-exp
 * weights -- the sequence-dimension KV partition of Section 5.2 -- through
 * the workspace.  The split depends only on the lengths and grid_blocks, and
 * pieces are merged in a fixed order, so repeated calls with the same inputs
 * give bitwise-identical results.
 *
 * Arguments (all device pointers, C-contiguous, row-major):
 *   q          [B, C_max, Hq, D] dtype.  Row (b, i) holds the queries of draft
 *              token i of sequence b; rows i >= c_b are never read.
 *   k_cache    [B, Hkv, S_max, D] dtype.  Rows [0, l_b) hold the cached
 *   v_cache    context, rows [l_b, l_b + c_b) the chunk's own keys/values,
 *              already appended.  Rows >= l_b + c_b are never read.
 *   ctx_lens   int32 [B]: l_b, the cached context length of sequence b.
 *   chunk_lens int32 [B]: c_b, the draft chunk length (gamma + 1) of b.
 *   scale      softmax scale applied to q.k (e.g. 1/sqrt(D)); finite and > 0
 *              (SPECMOE_ERR_SCALE otherwise).
 *   out        float32 [B, C_max, Hq, D]: attention output.
 *   lse        float32 [B, C_max, Hq]: natural-log log-sum-exp of the scaled,
 *              masked scores of each row.
 *   stream     hipStream_t the work is enqueued on (NULL: the null stream).
 *   desc       host pointer to the problem description.
 * Padding rows (c_b <= i < C_max) get out = 0 and lse = -inf.  A sequence with
 * c_b = 0 has only padding rows.
 *
 * Device-side preconditions (not checked on the host, since the lengths live
 * in device memory and the call never synchronises): 0 <= c_b <= C_max,
 * l_b >= 0, l_b + c_b <= S_max.  The kernels clamp violating lengths into
 * these ranges before any memory access, so a violation yields unspecified
 * values but never an out-of-bounds access.
 *
 * Ownership: the caller owns every buffer, including the workspace; the
 * library allocates nothing, keeps no pointer after returning, and does not
 * synchronise with the host: the work is asynchronous on `stream`, and the
 * buffers must stay valid until it completes.  Calls are reentrant; calls
 * that may run concurrently need distinct workspaces.  The workspace's
 * counter region must be zeroed once before its first call (see
 * specmoe_verify_attn_workspace_bytes); every call leaves it ready for the next.
 *
 * Errors: all host-side checks run before any HIP call; on an error nothing
 * is enqueued and one of the SPECMOE_ERR_* codes is returned.  A launch
 * failure reported by HIP returns SPECMOE_ERR_LAUNCH.  The waves of a
 * workgroup hand tiles to each other through bounded waits; a wait that
 * gives up (never expected: it means a broken hand-off) cannot be seen by
 * the asynchronous call itself, so it sets a sticky bit in the workspace,
 * which specmoe_verify_attn_status reports.
 */
int specmoe_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                        const int32_t* ctx_lens, const int32_t* chunk_lens,
                        float scale, float* out, float* lse, void* stream,
                        const specmoe_verify_desc* desc);

/*
 * specmoe_verify_attn_tree -- chunked verification attention for tree drafts.
 *
 * The same operation as specmoe_verify_attn, except inside the draft region:
 * when the draft tokens form a tree (Section 2.3: a tree of draft tokens is
 * verified as a sequence plus a mask relating them), the draft part of the
 * mask is given explicitly, and only that part (Section 5.1 stores only the
 * draft region of the mask; the cached part is always visible):
 *
 *   draft_mask  uint64 [B, C_max], device, 8-byte aligned.  Bit k of
 *               draft_mask[b * C_max + i] is set when draft token i of
 *               sequence b attends to draft token k, i.e. key position
 *               l_b + k.  Every cached key j < l_b is visible to every draft
 *               token.  Bits k >= c_b are ignored, words of rows i >= c_b are
 *               never read.  For a tree, word i holds the tokens on the path
 *               from the root to i (i included); a chain draft's word i is
 *               2^(i+1) - 1, which reproduces specmoe_verify_attn.  Any other
 *               bit pattern is allowed.
 *
 * A draft token that sees no key (l_b = 0 and no bit below c_b) gets out = 0
 * and lse = -inf, as a padding row does.  C_max must be <= 64
 * (SPECMOE_ERR_MASK otherwise); a NULL draft_mask is SPECMOE_ERR_NULL_POINTER
 * and a misaligned one SPECMOE_ERR_ALIGN (with B > 0).  Every other argument,
 * the workspace, the preconditions, ownership, determinism and the errors are
 * those of specmoe_verify_attn; the two entry points can share a workspace.
 */
int specmoe_verify_attn_tree(const void* q, const void* k_cache, const void* v_cache,
                             const int32_t* ctx_lens, const int32_t* chunk_lens,
                             const uint64_t* draft_mask, float scale, float* out, float* lse,
                             void* stream, const specmoe_verify_desc* desc);

/*
 * specmoe_verify_attn_noalloc -- specmoe_verify_attn for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * and harnesses that forbid hipMalloc.
 *
 * The same operation, arguments, layouts, preconditions, determinism and
 * errors as specmoe_verify_attn, except that desc->workspace and
 * desc->workspace_bytes are ignored: the kernels use a scratch array that
 * the library holds in static device memory, one per GPU (48 MiB, held until
 * the process ends), instead of a caller workspace.  Before the first call on
 * a device, its address is looked up once with that device current.  No call
 * allocates or frees anything (no hipMalloc, hipFree or allocating library
 * routine); each enqueues a small kernel that clears the scratch's arrival
 * counters, then the attention kernel, on `stream`.
 *
 * Limit: the workspace the descriptor needs
 * (specmoe_verify_attn_workspace_bytes) must fit in 48 MiB, which holds
 * every shape at the default grid; a larger need returns
 * SPECMOE_ERR_WORKSPACE before any HIP call.
 *
 * Every call on one GPU shares that GPU's scratch: calls that may overlap on
 * one GPU (on different streams, or from several host threads without
 * ordering) race and give unspecified results; serialise them, e.g. on one
 * stream.  A give-up of an in-kernel wait is recorded in the scratch's
 * status word, which specmoe_verify_attn_status(NULL, 0, stream) reads.
 */
int specmoe_verify_attn_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* ctx_lens, const int32_t* chunk_lens,
                                float scale, float* out, float* lse, void* stream,
                                const specmoe_verify_desc* desc);

/* Geometry of a paged KV cache (host struct). */
typedef struct specmoe_paged_kv {
  int32_t page_size;      /* tokens per page: a power of two in [8, 65536]            */
  int32_t pages_per_seq;  /* columns of the block table; desc->S_max must equal
                             page_size * pages_per_seq                               */
  int32_t num_pages;      /* pages in the pool                                        */
} specmoe_paged_kv;

/*
 * specmoe_verify_attn_paged -- chunked verification attention over a paged
 * KV cache.
 *
 * The operation of specmoe_verify_attn (or, with a draft_mask, of
 * specmoe_verify_attn_tree), with the KV cache held as a pool of pages
 * instead of one slab per sequence.  Paging is not part of the paper
 * (Section 2.2 only cites KV-cache managers); this layout is the library's:
 *
 *   k_pages, v_pages  [num_pages, Hkv, page_size, D] dtype, device, 16-byte
 *                aligned: page P holds page_size consecutive tokens of one
 *                sequence for every KV head.
 *   block_table  int32 [B, pages_per_seq], device: token j of sequence b is
 *                in page block_table[b * pages_per_seq + j / page_size], row
 *                j % page_size.  Only the entries that cover tokens
 *                [0, l_b + c_b) are read; an entry outside [0, num_pages) is
 *                clamped into it (unspecified values, never an out-of-bounds
 *                access).
 *   draft_mask   NULL for chain drafts, else as in specmoe_verify_attn_tree.
 *   paged        host pointer to the page geometry.
 *
 * Every other argument, the workspace, the preconditions (with
 * S_max = page_size * pages_per_seq), ownership, determinism and the errors
 * are those of specmoe_verify_attn; SPECMOE_ERR_PAGES reports a bad geometry,
 * SPECMOE_ERR_NULL_POINTER a NULL paged or (with B > 0) block_table.
 */
int specmoe_verify_attn_paged(const void* q, const void* k_pages, const void* v_pages,
                              const int32_t* block_table, const int32_t* ctx_lens,
                              const int32_t* chunk_lens, const uint64_t* draft_mask, float scale,
                              float* out, float* lse, void* stream, const specmoe_verify_desc* desc,
                              const specmoe_paged_kv* paged);

/* Bytes of device workspace specmoe_verify_attn needs for `desc` (its
 * grid_blocks included); 0 for an invalid descriptor.  The workspace starts
 * with a zeroed region -- a 256-byte header holding the sticky status word,
 * then one arrival counter per (sequence, KV head) of a launch of up to 1024
 * sequences, at offsets that depend only on Hkv -- followed by the partial
 * results of pieces (two slots per workgroup).  The zeroed region must be
 * zero before the first call; every call that completes leaves the counters
 * zero again (the workgroup that merges a unit resets its counter), so a
 * workspace initialised once by specmoe_verify_attn_workspace_init can be
 * reused for any number of calls with the same Hkv, any B, lengths and
 * grid_blocks, as long as it is large enough for them. */
size_t specmoe_verify_attn_workspace_bytes(const specmoe_verify_desc* desc);

/* Zero the zeroed region (status word and counters) of `workspace` (device,
 * workspace_bytes long) with a small kernel on `stream` (a hipStream_t; NULL:
 * the null stream); this also clears a recorded give-up.  Status:
 * SPECMOE_OK, a descriptor error, SPECMOE_ERR_NULL_POINTER, SPECMOE_ERR_ALIGN,
 * SPECMOE_ERR_WORKSPACE if the buffer is too small, or SPECMOE_ERR_LAUNCH. */
int specmoe_verify_attn_workspace_init(void* workspace, size_t workspace_bytes, void* stream,
                                       const specmoe_verify_desc* desc);

/* Status of the calls made so far with `workspace` (device, workspace_bytes
 * long, 16-byte aligned): SPECMOE_ERR_HANDOFF if a kernel's wait for another
 * wave gave up in any call since the workspace was last initialised, else
 * SPECMOE_OK.  Copies the 4-byte status word to the host on `stream` (a
 * hipStream_t; NULL: the null stream) and synchronises with that stream, so
 * it reports every call enqueued on it before; the word stays set until
 * specmoe_verify_attn_workspace_init clears it.  After SPECMOE_ERR_HANDOFF
 * the workspace must be initialised again before its next call: a give-up
 * can also leave arrival counters set.  workspace = NULL with
 * workspace_bytes = 0 reads the status word of the current device's static
 * scratch (specmoe_verify_attn_noalloc), which stays set until the process
 * ends.  SPECMOE_ERR_NULL_POINTER,
 * SPECMOE_ERR_ALIGN, SPECMOE_ERR_WORKSPACE (fewer than 256 bytes) or
 * SPECMOE_ERR_LAUNCH (HIP reported an error for the copy) otherwise. */
int specmoe_verify_attn_status(const void* workspace, size_t workspace_bytes, void* stream);

/* Keys per tile for `desc`'s dtype and D (32 KB of K rows).  Negative status
 * for an invalid dtype or D. */
int32_t specmoe_verify_attn_key_tile(const specmoe_verify_desc* desc);

/* Static, human-readable text for a status code. */
const char* specmoe_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* SPECMOE_VERIFY_H */
