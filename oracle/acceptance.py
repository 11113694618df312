"""Plain CPU oracle of the acceptance step that follows verification.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test-suite, the smoke
check and the CPU-baseline leg of the benchmark may import or run this module.
It shares no code with the HIP path and imports nothing from it.

After the target model's forward pass over a chunk, the draft tokens are
verified against what the target itself would have produced (Section 2.3:
the target model checks the draft tokens in one pass; Section 4.2: the draft
model then updates its KV cache from the verification result; Section 5.3
counts the verification among the per-iteration overheads).  The
chunk of sequence b holds c_b tokens: position 0 is the last token already
accepted, positions 1..c_b-1 are the draft tokens (a chunk of 1 is plain
decoding).  The logits at position i are the target's prediction for the
token at position i+1.

Readings where the paper is silent: verification is greedy -- the target's
prediction is the argmax of its logits (the lowest token id among equal
maxima), and a draft token is accepted when it equals the prediction at the
position before it and every earlier draft token was accepted.  With a
accepted draft tokens, the target's prediction after the last accepted token
(position a) is the next token, and the first a+1 chunk tokens -- the last
accepted token and the a accepted drafts -- have become context: the context
length grows from l_b to l_b + a + 1.  Rows of rejected draft tokens are simply
overwritten by the next chunk.  A sequence with c_b = 0 takes no step:
accepted 0, next token -1, context length unchanged, every argmax -1.

Parity pins (tests/test_oracle.py): brute force with pure-Python loops over
tiny inputs, planted maxima with known acceptance lengths, exact ties, the
chunk-of-1 case (plain greedy decoding), and the invariants that tie the
outputs together; planted mistakes in copies of this module are caught.
"""
from __future__ import annotations

import numpy as np

from .reference import to_f64


def greedy_argmax(row: np.ndarray) -> int:
    """Index of the largest value of a float64 row; the lowest index among
    equal maxima (numpy's argmax returns the first occurrence)."""
    return int(np.argmax(row))


def accept_greedy_ref(logits, draft_tokens, ctx_lens, chunk_lens, dtype: str):
    """Greedy acceptance of a batch of chunks.

    logits        [B, C_max, V]  target logits per chunk position ("bf16" as
                                  uint16 bit patterns, or "f32")
    draft_tokens  [B, C_max]     chunk token ids: position 0 the last accepted
                                  token, positions 1..c_b-1 the drafts
    ctx_lens, chunk_lens  [B]    l_b and c_b before the step

    Returns a dict of int64 arrays: argmax [B, C_max] (-1 past c_b), accepted
    [B] (a_b, draft tokens accepted), next_token [B] (the target's prediction
    after the last accepted token) and new_ctx_lens [B] (l_b + a_b + 1).
    """
    B, C_max, _ = logits.shape
    argmax = np.full((B, C_max), -1, np.int64)
    accepted = np.zeros(B, np.int64)
    next_token = np.full(B, -1, np.int64)
    new_ctx = np.asarray(ctx_lens, np.int64).copy()
    for b in range(B):
        c = int(chunk_lens[b])
        if c == 0:
            continue
        for i in range(c):
            argmax[b, i] = greedy_argmax(to_f64(logits[b, i], dtype))
        a = 0
        while a < c - 1 and argmax[b, a] == int(draft_tokens[b, a + 1]):
            a += 1
        accepted[b] = a
        next_token[b] = argmax[b, a]
        new_ctx[b] = int(ctx_lens[b]) + a + 1
    return dict(argmax=argmax, accepted=accepted, next_token=next_token, new_ctx_lens=new_ctx)


def tree_parent(words, i: int) -> int:
    """Parent of draft token i >= 1 in a tree given by root-path words (word i
    holds i and its ancestors): the highest ancestor bit below i."""
    rest = int(words[i]) & ~(1 << i) & ((1 << i) - 1)
    return rest.bit_length() - 1


def accept_tree_ref(logits, draft_tokens, draft_mask, ctx_lens, chunk_lens, dtype: str):
    """Greedy acceptance of tree drafts (Section 2.3: a tree of draft tokens
    is verified as a sequence plus a mask relating them).

    The chunk's tokens are the tree's nodes in topological order: node 0 is
    the last accepted token (the root), node i >= 1 a draft whose parent is
    given by the root-path words ``draft_mask`` [B, C_max] (word i: the bits
    of i and its ancestors, as in tree_mask).  Reading, as for chains: node i
    is accepted when its parent is and its token equals the target's
    prediction at the parent (the argmax of the parent's logits).  The
    deepest accepted node wins (the lowest index among equally deep ones);
    its root path is the accepted path, a = its depth, the next token is the
    prediction at it, and the context grows to l + a + 1.

    Returns the dict of accept_greedy_ref plus ``path`` [B] (int): the bit
    word of the accepted path (node indices; 0 when c_b = 0).
    """
    B, C_max, _ = logits.shape
    argmax = np.full((B, C_max), -1, np.int64)
    accepted = np.zeros(B, np.int64)
    next_token = np.full(B, -1, np.int64)
    new_ctx = np.asarray(ctx_lens, np.int64).copy()
    path = np.zeros(B, dtype=object)
    for b in range(B):
        c = int(chunk_lens[b])
        if c == 0:
            path[b] = 0
            continue
        for i in range(c):
            argmax[b, i] = greedy_argmax(to_f64(logits[b, i], dtype))
        ok = [True] + [False] * (c - 1)
        for i in range(1, c):
            par = tree_parent(draft_mask[b], i)
            ok[i] = ok[par] and argmax[b, par] == int(draft_tokens[b, i])
        depth = [bin(int(draft_mask[b][i]) & ((1 << c) - 1)).count("1") - 1 for i in range(c)]
        best = max((i for i in range(c) if ok[i]), key=lambda i: (depth[i], -i))
        accepted[b] = depth[best]
        next_token[b] = argmax[b, best]
        new_ctx[b] = int(ctx_lens[b]) + depth[best] + 1
        path[b] = int(draft_mask[b][best]) & ((1 << c) - 1)
    return dict(argmax=argmax, accepted=accepted, next_token=next_token, new_ctx_lens=new_ctx, path=path)


def compact_path_ref(cache, ctx_lens, path_words):
    """The KV cache after a tree acceptance: for every sequence b and KV head,
    the rows of the accepted path's nodes (rows l_b + k for the set bits k of
    the path word, ascending) move to rows l_b + 0, 1, ...; every other row
    keeps its value.  ``cache`` is [B, Hkv, S_max, D]; a copy is returned."""
    out = np.array(cache, copy=True)
    for b in range(out.shape[0]):
        l = int(ctx_lens[b])
        nodes = [k for k in range(64) if (int(path_words[b]) >> k) & 1]
        for j, k in enumerate(nodes):
            out[b, :, l + j] = cache[b, :, l + k]
    return out
