// Greedy acceptance of draft tokens for MI355X (gfx950, CDNA4).
//
// After verification, every chunk position's logits are reduced to their
// argmax (the target's prediction), and the leading drafts that match the
// prediction before them are accepted (SpecMoEOff, Section 2.3; the rule is
// greedy verification).  The work is a read of the logits, HBM-bound:
//   * the logits of the valid rows form a list of items (`split` vocabulary
//     entries of one row, 8 KB by default); a persistent grid of waves (two
//     workgroups of 8 waves per CU) takes contiguous ranges of the list, so
//     few workgroups are dispatched whatever the batch;
//   * a wave streams its items with 16-byte non-temporal loads, 4 KB per
//     wave in flight (every logit is read once), keeps a per-lane (max,
//     first index), and reduces it across the wave only where its range
//     leaves a row: one partial result per (row, wave) segment;
//   * after its last segment of a sequence, a wave counts itself on an LDS
//     counter of its workgroup; the workgroup's last wave for the sequence
//     counts the workgroup on the sequence's arrival counter (device-scope
//     atomics on one address serialise, so one per workgroup rather than one
//     per wave); the last to arrive combines the segments in vocabulary
//     order, decides the acceptance with one ballot per 64 chunk positions
//     and writes the sequence's outputs -- one launch, no host step.
#include <hip/hip_runtime.h>

#include <limits.h>
#include <math.h>
#include <stdint.h>

#include "specmoe_accept.h"

namespace {

constexpr int kWavesPerGroup = 8;
constexpr int kThreads = 64 * kWavesPerGroup;
constexpr int kGroupsPerCU = 2;
constexpr int kCUs = 256;                  // MI355X
constexpr int kVecBytes = 16;
constexpr int kItemBytes = 8192;           // default item: 8 KB of logits
// 16-byte loads per lane in flight (4 KB per wave): measured faster than 2,
// 8 or 16, and than issuing the next batch before reducing the current one
constexpr int kBatch = 4;
constexpr int kSplitUnit = 512;            // item granularity (entries)
constexpr int kMaxChunk = 1024;            // C_max limit
constexpr int kMaxSeqs = 65536;            // B limit (fixed counter region)
constexpr int kGroupSeqs = 16;             // sequences a workgroup counts through LDS
// Partial results go through, or around, the XCD-local L2 to where every XCD
// sees them (device scope), without an L2-wide write-back.
constexpr int kDeviceCoherent = 16;        // SC1
constexpr int kBufferFormat = 0x00020000;

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) int i32x2;

struct Params {
  const char* logits;
  const int32_t* tokens;
  const int32_t* ctx_lens;
  const int32_t* chunk_lens;
  int32_t* argmax;
  int32_t* accepted;
  int32_t* next_token;
  int32_t* new_ctx;
  int* counters;    // [kMaxSeqs] waves arrived per sequence, zero between calls
  char* part;       // [N] (max value bits, index) of the segment starting at each item
  int part_bytes;
  int B, C_max, V, S, split;
  int N;            // items: B * C_max * S
  int q;            // items per wave range
  int grouped;      // count arrivals per workgroup (every workgroup range meets < kGroupSeqs sequences)
  const uint64_t* draft_mask;   // tree drafts: [B][C_max] root-path words (NULL: chain drafts)
  uint64_t* path;               // tree drafts: [B] the accepted path's node bits
};

// (v, i) beats (bv, bi): a larger value, or an equal one at a lower index.
// Floating-point equality makes +0 and -0 equal; -inf rows still elect their
// first index because the starting index is INT_MAX.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// (max, first index) over the wave, returned in every lane
__device__ __forceinline__ void wave_best(float& bv, int& bi) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(bv, off);
    const int oi = __shfl_xor(bi, off);
    if (better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
}

template <bool BF16>
__global__ __launch_bounds__(kThreads, kGroupsPerCU) void accept_kernel(Params p) {
  constexpr int kElt = BF16 ? 2 : 4;
  constexpr int kPer = kVecBytes / kElt;   // entries per 16-byte vector
  __shared__ int group_cnt[kGroupSeqs];
  const int lane = threadIdx.x & 63;
  const int wave = uniform(blockIdx.x * kWavesPerGroup + (threadIdx.x >> 6));
  const int CS = p.C_max * p.S;            // items per sequence
  const int gq = kWavesPerGroup * p.q;     // items per workgroup range
  const int g0 = blockIdx.x * gq;
  const int g1 = min(g0 + gq, p.N);
  // sequences the workgroup's range meets: when no workgroup range meets
  // kGroupSeqs of them (the same choice for the whole grid, so that every
  // sequence expects the same kind of arrival), waves are counted in LDS first
  const int gb0 = g0 / CS;
  const bool grouped = p.grouped != 0;
  if (threadIdx.x < kGroupSeqs) group_cnt[threadIdx.x] = 0;
  __syncthreads();
  const int x0 = wave * p.q;
  const int x1 = min(x0 + p.q, p.N);
  if (x0 >= x1) return;
  const __amdgpu_buffer_rsrc_t part_rsrc = __builtin_amdgcn_make_buffer_rsrc(p.part, 0, p.part_bytes, kBufferFormat);

  for (int b = x0 / CS; b * CS < x1; ++b) {
    const int c = uniform(min(max(p.chunk_lens[b], 0), p.C_max));
    if (c == 0) {
      // no step; written by the wave that owns the sequence's first item
      if (b * CS >= x0) {
        for (int k = lane; k < p.C_max; k += 64) p.argmax[(size_t)b * p.C_max + k] = -1;
        if (lane == 0) {
          p.accepted[b] = 0;
          p.next_token[b] = -1;
          p.new_ctx[b] = p.ctx_lens[b];
          if (p.draft_mask) p.path[b] = 0;
        }
      }
      continue;
    }
    // this wave's items of the sequence's valid rows
    const int ya = max(x0, b * CS), yb = min(x1, b * CS + c * p.S);
    if (ya >= yb) continue;
    float bv = -INFINITY;
    int bi = INT_MAX;
    int seg = ya;                          // first item of the current row segment
    for (int y = ya; y < yb; ++y) {
      const int row = y / p.S;
      const int lo = (y - row * p.S) * p.split;
      const int nvec = (min(lo + p.split, p.V) - lo) / kPer;   // V and split are multiples of kPer
      const u32x4* src = reinterpret_cast<const u32x4*>(p.logits + ((size_t)row * p.V + lo) * kElt);
      for (int v0 = 0; v0 < nvec; v0 += 64 * kBatch) {
        u32x4 x[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int v = v0 + u * 64 + lane;
          x[u] = v < nvec ? __builtin_nontemporal_load(src + v) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int v = v0 + u * 64 + lane;
          if (v < nvec) {
            const int idx = lo + v * kPer;
#pragma unroll
            for (int e = 0; e < kPer; ++e) {
              float val;
              if constexpr (BF16) {
                // bf16 entry 2k is the low half of word k, 2k+1 the high half
                const uint32_t wd = x[u][e >> 1];
                val = __uint_as_float((e & 1) ? (wd & 0xffff0000u) : (wd << 16));
              } else {
                val = __uint_as_float(x[u][e]);
              }
              if (better(val, idx + e, bv, bi)) {
                bv = val;
                bi = idx + e;
              }
            }
          }
        }
      }
      if (y + 1 == yb || (y + 1) / p.S != row) {
        // the wave leaves this row: publish the segment's maximum
        wave_best(bv, bi);
        if (lane == 0)
          __builtin_amdgcn_raw_buffer_store_b64(i32x2{__float_as_int(bv), bi}, part_rsrc, seg * 8, 0,
                                                kDeviceCoherent);
        bv = -INFINITY;
        bi = INT_MAX;
        seg = y + 1;
      }
    }
    // what the sequence's last wave needs besides the segments is loaded now,
    // so that it rides the wait for the segment stores: the context length
    // and the draft tokens of the first 64 chunk positions
    const int l_b = p.ctx_lens[b];
    // chains: the draft after position lane; trees: node lane's own token
    // and root-path word
    const bool tree = p.draft_mask != nullptr;
    const int tok0 = tree ? (lane < c ? p.tokens[(size_t)b * p.C_max + lane] : -1)
                          : (lane < c - 1 ? p.tokens[(size_t)b * p.C_max + lane + 1] : -1);
    const uint64_t word0 = tree && lane < c ? p.draft_mask[(size_t)b * p.C_max + lane] : 0;
    // count this wave once its segments are stored
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const int first = b * CS, last = b * CS + c * p.S - 1;   // the sequence's valid items
    int arrivals;     // arrivals the sequence's counter expects
    bool counts = true;
    if (grouped) {
      // the workgroup's waves that meet the valid items count in LDS; the
      // last of them counts the workgroup
      const int fa = max(first, g0), la = min(last, g1 - 1);
      const int in_group = la / p.q - fa / p.q + 1;
      int old_l = 0;
      if (lane == 0) old_l = atomicAdd(&group_cnt[b - gb0], 1);
      counts = uniform(old_l) == in_group - 1;
      arrivals = last / gq - first / gq + 1;   // workgroups whose ranges meet the valid items
    } else {
      arrivals = last / p.q - first / p.q + 1;  // waves whose ranges meet the valid items
    }
    if (!counts) continue;
    int old = 0;
    if (lane == 0) old = __hip_atomic_fetch_add(p.counters + b, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    old = uniform(old);
    if (old != arrivals - 1) continue;

    // ---- the last wave of sequence b: predictions, then the acceptance
    int a = -1, next = -1, cand = -1;
    for (int k0 = 0; k0 < p.C_max; k0 += 64) {
      const int k = k0 + lane;
      int pred = -1;
      const int tok = k0 == 0 ? tok0 : (k < c - 1 ? p.tokens[(size_t)b * p.C_max + k + 1] : -1);
      if (k < c) {
        float rv = -INFINITY;
        int ri = INT_MAX;
        const int rs = (b * p.C_max + k) * p.S, re = rs + p.S - 1;
        const int w0 = rs / p.q, w1 = re / p.q;
        // the row's segments in vocabulary order, loaded kGather at a time
        constexpr int kGather = 8;
        for (int wb = w0; wb <= w1; wb += kGather) {
          i32x2 e[kGather];
#pragma unroll
          for (int u = 0; u < kGather; ++u) {
            const int slot = max(rs, (wb + u) * p.q);
            e[u] = wb + u <= w1 ? __builtin_bit_cast(i32x2, __builtin_amdgcn_raw_buffer_load_b64(
                                                                 part_rsrc, slot * 8, 0, kDeviceCoherent))
                                : i32x2{0, INT_MAX};
          }
#pragma unroll
          for (int u = 0; u < kGather; ++u)
            if (wb + u <= w1 && better(__int_as_float(e[u][0]), e[u][1], rv, ri)) {
              rv = __int_as_float(e[u][0]);
              ri = e[u][1];
            }
        }
        pred = ri == INT_MAX ? -1 : ri;   // (a row of NaN elects nothing)
      }
      if (k < p.C_max) p.argmax[(size_t)b * p.C_max + k] = pred;
      if (tree) {
        // (C_max <= 64: one pass) node k's parent is its highest ancestor
        // bit below k; the edge into k is rejected when k's token differs
        // from the parent's prediction, and a node is accepted when no edge
        // on its root path is.  The deepest accepted node wins, the lowest
        // index among equally deep ones.
        const uint64_t cmask = c >= 64 ? ~0ull : (1ull << c) - 1;
        const uint64_t word = word0 & cmask;
        const uint64_t above = word & ((1ull << k) - 1);
        const int par = above ? 63 - __builtin_clzll(above) : -1;
        const int ppred = __shfl(pred, par & 63);
        const bool reject = k >= 1 && k < c && (par < 0 || tok != ppred);
        const uint64_t rejected = __ballot(reject);
        const bool ok = k < c && (word & rejected) == 0;
        int key = ok ? ((__popcll(word) - 1) << 8) | (255 - k) : -1;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) key = max(key, __shfl_xor(key, off));
        const int d = 255 - (key & 255);
        a = key >> 8;
        next = __shfl(pred, d);
        const uint32_t path_lo = (uint32_t)__shfl((int)(uint32_t)word, d);
        const uint32_t path_hi = (uint32_t)__shfl((int)(uint32_t)(word >> 32), d);
        if (lane == 0) p.path[b] = ((uint64_t)path_hi << 32) | path_lo;
        break;
      }
      // draft k + 1 is rejected when it differs from prediction k
      const bool reject = k < c - 1 && tok != pred;
      const uint64_t m = __ballot(reject);
      const int first_reject = m ? (int)__builtin_ctzll(m) : 64;
      const int at_reject = __shfl(pred, first_reject & 63);
      const int at_end = __shfl(pred, (c - 1 - k0) & 63);
      if (a < 0 && m) {
        a = k0 + first_reject;
        next = at_reject;
      }
      if (c - 1 >= k0 && c - 1 < k0 + 64) cand = at_end;
    }
    if (a < 0) {
      a = c - 1;
      next = cand;
    }
    if (lane == 0) {
      p.accepted[b] = a;
      p.next_token[b] = next;
      p.new_ctx[b] = l_b + a + 1;
      __hip_atomic_store(p.counters + b, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);   // ready for the next call
    }
  }
}

// Move the accepted path's K (blockIdx.y = 0) or V (1) rows of one (sequence,
// KV head) (blockIdx.x) to the rows right after the context: row l + node_j
// to row l + j for the j-th set bit node_j of the path word.  Every row is
// read before any is written, so overlapping moves are safe.
constexpr int kCompactThreads = 256;
constexpr int kCompactChunks = 8;   // 16-byte chunks per thread: 64 rows of up to 512 bytes

__global__ __launch_bounds__(kCompactThreads) void compact_kernel(char* k, char* v, const int32_t* ctx_lens,
                                                                 const uint64_t* path, int Hkv, int S_max,
                                                                 int row_bytes) {
  const int unit = blockIdx.x;
  const int b = unit / Hkv;
  char* slab = (blockIdx.y == 0 ? k : v) + (size_t)unit * S_max * row_bytes;
  const int l = min(max(ctx_lens[b], 0), S_max);
  const uint64_t w = path[b];
  const int chunks = row_bytes / 16;
  const int n = __popcll(w);
  u32x4 buf[kCompactChunks];
  int dst[kCompactChunks];
#pragma unroll
  for (int u = 0; u < kCompactChunks; ++u) {
    const int t = threadIdx.x + u * kCompactThreads;
    const int j = t / chunks;
    dst[u] = -1;
    if (j < n) {
      uint64_t rest = w;   // the j-th set bit: clear j lowest set bits
      for (int i = 0; i < j; ++i) rest &= rest - 1;
      const int node = __builtin_ctzll(rest);
      const int ch = t - j * chunks;
      if (node != j && l + node < S_max) {
        buf[u] = *reinterpret_cast<const u32x4*>(slab + (size_t)(l + node) * row_bytes + 16 * ch);
        dst[u] = (l + j) * row_bytes + 16 * ch;
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kCompactChunks; ++u)
    if (dst[u] >= 0) *reinterpret_cast<u32x4*>(slab + dst[u]) = buf[u];
}

__global__ void zero_kernel(int* x, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] = 0;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

int elt_of(const specmoe_accept_desc* d) { return d->dtype == SPECMOE_BF16 ? 2 : 4; }

int split_of(const specmoe_accept_desc* d) { return d->split ? d->split : kItemBytes / elt_of(d); }

int validate(const specmoe_accept_desc* d) {
  if (!d) return SPECMOE_ERR_NULL_POINTER;
  if (d->dtype != SPECMOE_F32 && d->dtype != SPECMOE_BF16) return SPECMOE_ERR_DTYPE;
  if (d->flags != 0) return SPECMOE_ERR_FLAGS;
  if (d->B < 0 || d->B > kMaxSeqs || d->C_max < 1 || d->C_max > kMaxChunk || d->V < 1) return SPECMOE_ERR_SHAPE;
  const int64_t elt = elt_of(d);
  if ((d->V * elt) % kVecBytes != 0) return SPECMOE_ERR_SHAPE;
  if (d->split < 0 || d->split % kSplitUnit != 0) return SPECMOE_ERR_SHAPE;
  const int64_t S = (d->V + (int64_t)split_of(d) - 1) / split_of(d);
  // row offsets in elements, item indices and partial offsets in bytes stay
  // in 32 bits
  if ((int64_t)d->B * d->C_max * d->V >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  if ((int64_t)d->B * d->C_max * S * 8 >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  return SPECMOE_OK;
}

struct Plan {
  int S, N, q, groups, grouped;
  size_t counter_bytes, part_off, bytes;
};

Plan make_plan(const specmoe_accept_desc* d) {
  Plan pl;
  pl.S = (d->V + split_of(d) - 1) / split_of(d);
  pl.N = d->B * d->C_max * pl.S;
  // contiguous ranges of q items for at most the persistent grid's waves
  const int waves = kCUs * kGroupsPerCU * kWavesPerGroup;
  pl.q = pl.N > 0 ? (pl.N + waves - 1) / waves : 1;
  const int used = pl.N > 0 ? (pl.N + pl.q - 1) / pl.q : 0;
  pl.groups = (used + kWavesPerGroup - 1) / kWavesPerGroup;
  // a range of gq items meets at most (gq - 1) / CS + 2 sequences
  const int64_t gq = (int64_t)kWavesPerGroup * pl.q, CS = (int64_t)d->C_max * pl.S;
  pl.grouped = (gq - 1) / CS + 2 <= kGroupSeqs;
  pl.counter_bytes = align256((size_t)kMaxSeqs * sizeof(int));
  pl.part_off = pl.counter_bytes;
  pl.bytes = pl.part_off + (size_t)pl.N * 8;
  return pl;
}

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

int accept_run(const void* logits, const int32_t* tokens, const uint64_t* draft_mask, const int32_t* ctx_lens,
               const int32_t* chunk_lens, int32_t* argmax, int32_t* accepted, int32_t* next_token,
               int32_t* new_ctx_lens, uint64_t* path, void* stream, const specmoe_accept_desc* desc) {
  const int st = validate(desc);
  if (st != SPECMOE_OK) return st;
  if (desc->B == 0) return SPECMOE_OK;
  if (!logits || !tokens || !ctx_lens || !chunk_lens || !argmax || !accepted || !next_token || !new_ctx_lens)
    return SPECMOE_ERR_NULL_POINTER;
  if (!aligned16(logits)) return SPECMOE_ERR_ALIGN;
  const Plan pl = make_plan(desc);
  if (!desc->workspace) return SPECMOE_ERR_NULL_POINTER;
  if (!aligned16(desc->workspace)) return SPECMOE_ERR_ALIGN;
  if (desc->workspace_bytes < pl.bytes) return SPECMOE_ERR_WORKSPACE;

  Params p;
  p.logits = static_cast<const char*>(logits);
  p.tokens = tokens;
  p.ctx_lens = ctx_lens;
  p.chunk_lens = chunk_lens;
  p.argmax = argmax;
  p.accepted = accepted;
  p.next_token = next_token;
  p.new_ctx = new_ctx_lens;
  char* ws = static_cast<char*>(desc->workspace);
  p.counters = reinterpret_cast<int*>(ws);
  p.part = ws + pl.part_off;
  p.part_bytes = (int)(pl.bytes - pl.part_off);
  p.B = desc->B;
  p.C_max = desc->C_max;
  p.V = desc->V;
  p.S = pl.S;
  p.split = split_of(desc);
  p.N = pl.N;
  p.q = pl.q;
  p.grouped = pl.grouped;
  p.draft_mask = draft_mask;
  p.path = path;
  const unsigned grid = (unsigned)pl.groups;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (desc->dtype == SPECMOE_BF16)
    hipLaunchKernelGGL(accept_kernel<true>, dim3(grid), dim3(kThreads), 0, s, p);
  else
    hipLaunchKernelGGL(accept_kernel<false>, dim3(grid), dim3(kThreads), 0, s, p);
  return hipGetLastError() == hipSuccess ? SPECMOE_OK : SPECMOE_ERR_LAUNCH;
}

}  // namespace

extern "C" {

size_t specmoe_accept_workspace_bytes(const specmoe_accept_desc* desc) {
  if (validate(desc) != SPECMOE_OK) return 0;
  return make_plan(desc).bytes;
}

int specmoe_accept_workspace_init(void* workspace, size_t workspace_bytes, void* stream,
                                  const specmoe_accept_desc* desc) {
  const int st = validate(desc);
  if (st != SPECMOE_OK) return st;
  if (!workspace) return SPECMOE_ERR_NULL_POINTER;
  if (!aligned16(workspace)) return SPECMOE_ERR_ALIGN;
  const Plan pl = make_plan(desc);
  if (workspace_bytes < pl.bytes) return SPECMOE_ERR_WORKSPACE;
  const int n = (int)(pl.counter_bytes / sizeof(int));
  (void)hipGetLastError();
  hipLaunchKernelGGL(zero_kernel, dim3((n + 255) / 256), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<int*>(workspace), n);
  return hipGetLastError() == hipSuccess ? SPECMOE_OK : SPECMOE_ERR_LAUNCH;
}

int specmoe_accept_greedy(const void* logits, const int32_t* tokens, const int32_t* ctx_lens,
                          const int32_t* chunk_lens, int32_t* argmax, int32_t* accepted, int32_t* next_token,
                          int32_t* new_ctx_lens, void* stream, const specmoe_accept_desc* desc) {
  return accept_run(logits, tokens, nullptr, ctx_lens, chunk_lens, argmax, accepted, next_token, new_ctx_lens,
                    nullptr, stream, desc);
}

int specmoe_accept_greedy_tree(const void* logits, const int32_t* tokens, const uint64_t* draft_mask,
                               const int32_t* ctx_lens, const int32_t* chunk_lens, int32_t* argmax,
                               int32_t* accepted, int32_t* next_token, int32_t* new_ctx_lens, uint64_t* path,
                               void* stream, const specmoe_accept_desc* desc) {
  if (desc && validate(desc) == SPECMOE_OK && desc->C_max > 64) return SPECMOE_ERR_MASK;
  if (desc && desc->B > 0 && (!draft_mask || !path)) return SPECMOE_ERR_NULL_POINTER;
  if ((reinterpret_cast<uintptr_t>(draft_mask) & 7u) || (reinterpret_cast<uintptr_t>(path) & 7u))
    return SPECMOE_ERR_ALIGN;
  return accept_run(logits, tokens, draft_mask, ctx_lens, chunk_lens, argmax, accepted, next_token, new_ctx_lens,
                    path, stream, desc);
}

int specmoe_compact_accepted_kv(void* k_cache, void* v_cache, const int32_t* ctx_lens, const uint64_t* path,
                                void* stream, const specmoe_verify_desc* desc) {
  if (!desc) return SPECMOE_ERR_NULL_POINTER;
  if (desc->dtype != SPECMOE_F32 && desc->dtype != SPECMOE_BF16 && desc->dtype != SPECMOE_F16)
    return SPECMOE_ERR_DTYPE;
  if (desc->D != 64 && desc->D != 128) return SPECMOE_ERR_HEAD_DIM;
  if (desc->B < 0 || desc->Hkv <= 0 || desc->S_max < 1) return SPECMOE_ERR_SHAPE;
  const int64_t row_bytes = (int64_t)desc->D * (desc->dtype == SPECMOE_F32 ? 4 : 2);
  if ((int64_t)desc->S_max * row_bytes >= ((int64_t)1 << 31) || (int64_t)desc->B * desc->Hkv >= (1 << 30))
    return SPECMOE_ERR_SHAPE;
  if (desc->B == 0) return SPECMOE_OK;
  if (!k_cache || !v_cache || !ctx_lens || !path) return SPECMOE_ERR_NULL_POINTER;
  if (!aligned16(k_cache) || !aligned16(v_cache) || (reinterpret_cast<uintptr_t>(path) & 7u))
    return SPECMOE_ERR_ALIGN;
  (void)hipGetLastError();
  hipLaunchKernelGGL(compact_kernel, dim3(desc->B * desc->Hkv, 2), dim3(kCompactThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<char*>(k_cache), static_cast<char*>(v_cache),
                     ctx_lens, path, desc->Hkv, desc->S_max, (int)row_bytes);
  return hipGetLastError() == hipSuccess ? SPECMOE_OK : SPECMOE_ERR_LAUNCH;
}

}  // extern "C"
