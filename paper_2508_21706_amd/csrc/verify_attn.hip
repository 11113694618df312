// Chunked verification attention for MI355X (gfx950, CDNA4).
//
// Computes, for every sequence b and KV head, softmax(scale*Q K^T + M) V over
// the cached context plus the draft chunk, with a chain mask inside the chunk
// or, for tree drafts, per-token draft-mask words (SpecMoEOff, Section 5.1,
// Section 2.3), and the log-sum-exp of every row.  The KV cache is one slab
// per sequence or a pool of pages found through a block table; elements are
// f32, bf16 or f16.
//
// Design (one kernel launch per call, one persistent workgroup per CU):
//   * Unit of work = (sequence b, KV head).  The c_b draft tokens times the g
//     query heads that share the KV head form the unit's R_b = c_b*g query
//     rows, cut into 16-row blocks, so that Q K^T and P V become small dense
//     MFMA contractions that reuse every K/V byte for all rows.
//   * Key tiles: a unit's keys [0, T_b) are cut into tiles of 32 KB of K rows
//     anchored at T_b (tile n-1 = [T_b - kTileKeys, T_b)), so the chunk's own
//     keys sit at the end of the unit's last tile.
//   * Stream-K schedule: the tiles of all units, in unit order, form one list
//     cut into contiguous ranges of equal cost, one per workgroup.  A tile's
//     cost grows with its unit's row count (a unit with many rows computes
//     longer on a tile than the tile takes to stream); when every unit has
//     the same rows, every workgroup streams the same number of K/V bytes.
//     The first tile of every workgroup is located by a search of per-sequence
//     prefix sums in LDS, computed by one wave of each workgroup from the
//     length arrays while the others wait at a single barrier, so no host
//     pass or second launch is needed.  A unit cut by a range
//     boundary is a sequence-wise KV partition whose partial results must be
//     combined, as the paper notes for its sequence-dimension KV split
//     (Section 5.2).  Ranges are streamed in order.  The piece of a range's
//     first segment is written as (O/l, lse) to the workspace and counted on
//     the unit's arrival counter; the piece of its last segment stays in
//     registers, and after its tiles the range merges it with log-sum-exp
//     weights with the next range's piece, when that is the unit's only
//     other piece and has arrived.  Other cut units are merged from the
//     workspace after the tiles of the last piece to arrive or of the first
//     holder to finish.
//   * Warp-specialised pipeline: 4 producer waves stream K/V tiles from HBM
//     straight into LDS with direct-to-LDS loads (one wave instruction moves
//     1 KB of contiguous cache rows); 8 consumer waves compute.  The producers
//     form two pairs, each owning one of two LDS stages; tiles and stages are
//     handed over through LDS counters (no workgroup barrier on the tile
//     path), so one pair's tile is in flight while the other's is computed.
//     Only the producers issue tile loads, so a consumer's wait for its own
//     stores or loads never drains the tile stream.  Staged K rows are padded
//     by 16 bytes and (bf16, D = 128) V rows by 32, so the score operand
//     reads and the transposed V reads are free of bank conflicts, and all
//     operand addresses are a per-lane base plus an immediate.
//   * Scores are formed transposed, S^T = K Q^T (keys on the MFMA M side,
//     query rows on N), so each lane holds one query row and four keys: row
//     statistics need two cross-lane steps, and the probabilities are already
//     the B operand of O^T = V^T P^T.  A consumer wave takes two 16-key blocks
//     of a tile; the waves that share a row block merge their partial (max,
//     sum, O) states through LDS at the end of each unit.
//   * bf16 (f16) inputs use v_mfma_f32_16x16x32_bf16 (_f16) for the scores
//     and for P V (one 32-key contraction over the wave's two blocks), with
//     fp32 accumulation (P is rounded to the input type for the PV product);
//     f32 inputs use v_mfma_f32_16x16x4_f32.  The two 16-bit types share
//     every layout and differ only in these instructions.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "specmoe_verify.h"

// Device scratch of specmoe_verify_attn_noalloc (for callers that cannot
// allocate): the workspace layout of a normal call (header, arrival
// counters, partial results) in one file-scope array per GPU, held until the
// process ends.  Host code never passes the array's name to a kernel (on the
// host it is only a stand-in for the symbol): it uses the device address
// that hipGetSymbolAddress returns for the current device.
constexpr size_t kScratchBytes = (size_t)48 << 20;
static __device__ __attribute__((aligned(256))) char scratch[kScratchBytes];

namespace {

constexpr int kProducers = 4;                 // waves that stream K/V into LDS
constexpr int kConsumers = 8;                 // waves that compute
constexpr int kWaves = kProducers + kConsumers;
constexpr int kThreads = 64 * kWaves;
constexpr int kCThreads = 64 * kConsumers;
constexpr int kStages = 2;                    // LDS stages: one per producer pair
constexpr int kHalf = 32768;                  // K bytes (and V bytes) of one tile
constexpr int kMaxDma = 18;                   // DMA instructions per producer wave and K (or V) tile, at most
constexpr int kBlk = 16;                      // keys (and query rows) per MFMA block
constexpr int kMaxRows = 128;                 // row blocks per unit <= 8
constexpr int kDefaultGrid = 256;             // persistent workgroups: one per CU of an MI355X
constexpr int kMaxGrid = 2048;
constexpr int kMaxSeqs = 1024;                // sequences per launch (their lengths live in LDS)
constexpr int kMaxDraftBits = 64;             // draft tokens a draft-mask word covers
constexpr float kLog2e = 1.4426950408889634f;
// The running max is only raised when a block's max exceeds it by more than
// this (log2 units): probabilities stay <= 2^8, and the O rescale is skipped
// for most blocks.
constexpr float kLazyMax = 8.f;
constexpr float kLn2 = 0.6931471805599453f;


typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;

// Element types of q, k and v (the specmoe_dtype codes)
constexpr int kF32 = SPECMOE_F32, kBF16 = SPECMOE_BF16, kF16 = SPECMOE_F16;
typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(4))) int i32x4;

// Cache policy of the partial-result accesses: device (agent) scope, so the
// data goes through, or around, the XCD-local L2 to the point where every XCD
// sees it, without an L2-wide write-back or invalidate.
constexpr int kDeviceCoherent = 16;   // SC1
// Cache policy of the K/V tile loads: non-temporal (NT).  Every K/V byte is
// read once, so the stream should not displace the cache lines that are
// reused (the partial results, the output being written); with the default
// policy the whole launch ran 6-11% slower.
constexpr int kStreaming = 2;
// kernel variants (template argument MODE)
constexpr int kModePlain = 0, kModeHold = 1, kModeNt = 2;
constexpr int kBufferFormat = 0x00020000;   // raw 32-bit buffer descriptor word 3

struct Params {
  const char* q;
  const char* k;
  const char* v;
  const int32_t* ctx_lens;
  const int32_t* chunk_lens;
  float* out;
  float* lse;
  int* status;      // sticky flags of the workspace: kGaveUp once an in-kernel wait gave up
  int spin_limit;   // polls before an in-kernel wait gives up
  int* counters;    // [B*Hkv] pieces arrived per unit (| kClaimed once a merge is claimed), zero between calls
  float* ws_o;      // [2P][Rcap][D] normalised partial outputs
  float* ws_lse;    // [2P][Rcap] partial log-sum-exp
  int ws_o_bytes, ws_lse_bytes;
  int B, Hq, Hkv, g, C_max, S_max;
  int Rcap;         // C_max * g
  int P;            // persistent workgroups
  float sl2;        // scale * log2(e)
  const uint64_t* draft_mask;   // [B][C_max] draft-mask words (tree drafts only)
  // paged caches only: k and v are [num_pages][Hkv][1 << page_shift][D]
  const int32_t* block_table;   // [B][pages_per_seq]
  int page_shift, pages_per_seq, num_pages;
};

// W16: 16-bit elements (bf16 or f16), which share every layout
template <bool W16, int D>
struct Cfg {
  static constexpr int kElt = W16 ? 2 : 4;
  static constexpr int kRowBytes = D * kElt;
  static constexpr int kChunks = kRowBytes / 16;           // 16-byte chunks per row
  static constexpr int kTileKeys = kHalf / kRowBytes;
  // LDS slots per staged row: the chunks and pad slots.  K rows carry one
  // pad (a 16-byte shift per row: the 16 rows of a score operand read sit in
  // distinct banks).  bf16 D = 128 V rows carry two (a 32-byte shift: the
  // transposed V reads take 4 rows x 32 bytes per 16 lanes, which one pad
  // would leave two-way bank conflicted); other layouts keep one.
  static constexpr int kSlotsK = kChunks + 1;
  static constexpr int kSlotsV = kChunks + (W16 && D == 128 ? 2 : 1);
  static constexpr int kPitchK = 16 * kSlotsK;              // padded LDS row pitches
  static constexpr int kPitchV = 16 * kSlotsV;
  static constexpr int kLdsK = kTileKeys * kPitchK;         // LDS bytes of a staged K (V) tile
  static constexpr int kLdsV = kTileKeys * kPitchV;
  static constexpr int kStage = kLdsK + kLdsV;
  static constexpr int kInstK = (kTileKeys * kSlotsK + 63) / 64;   // 64-slot DMA instructions per K (V) tile
  static constexpr int kInstV = (kTileKeys * kSlotsV + 63) / 64;
  static constexpr int kNKB = kTileKeys / kBlk;             // 16-key blocks per tile
  static constexpr int kDB = D / 16;                        // 16-wide d blocks of O^T
  static constexpr int kQJ = kChunks / 4;                   // 16-byte Q chunks per lane
  static_assert(kInstK <= 2 * kMaxDma && kInstV <= 2 * kMaxDma, "DMA instructions per producer wave");
  // LDS beside the stages: packed lengths and tile prefix sums of up to
  // kMaxSeqs sequences, the key-split merge statistics and the hand-off words
  static constexpr int kLdsFixed = kMaxSeqs * 4 + (kMaxSeqs + 1) * 4 + kConsumers * 2 * kBlk * 4 + 512;
  // the rest of the 160 KB: the cost prefix sums while the schedule is made,
  // then the piece of the range's first segment until the range's last tile
  static constexpr int kPieceLds = (160 * 1024 - kStages * kStage - kLdsFixed) / 16 * 16;
  static_assert(kPieceLds >= (kMaxSeqs + 1) * 4, "LDS budget");
  static_assert(kConsumers * 64 * D <= kStage, "key-split merge scratch fits in a stage");
  // the most (row block, key slot) regions a merge uses: one block with
  // min(kConsumers, kNKB / 2) key slots, or two blocks with two each
  static constexpr int kMergeRegions = kConsumers < kNKB / 2 ? kConsumers : kNKB / 2 > 4 ? kNKB / 2 : 4;
  static_assert(kMergeRegions * 64 * D <= kLdsK, "key-split merge scratch stays in the K half of a stage");
  static_assert(kNKB >= 2, "key blocks are processed in pairs");
};

// Hand-offs between the waves of a workgroup go through LDS counters that
// only grow: a wave adds one when it has done its part, and a waiting wave
// polls until the counter reaches the total it needs.  The wait is bounded
// (about 0.1 s of polling by default), so that a broken hand-off ends the
// kernel instead of hanging the GPU; a wait that gives up returns false, and
// the kernel then raises the sticky give-up flag in the workspace.  With a
// limit of 0 the counter is checked once.
constexpr int kSpinLimit = 1 << 21;
constexpr int kGaveUp = 1;   // status-word bit: an in-kernel wait gave up
constexpr int kClaimed = 1 << 30;   // unit counter bit: a holder has claimed the unit's merge
__device__ __forceinline__ bool wait_count(int* c, int target, int limit) {
  for (int spin = 0;; ++spin) {
    if (__builtin_amdgcn_readfirstlane(__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) >= target) {
      asm volatile("" ::: "memory");
      return true;
    }
    if (spin >= limit) break;
    __builtin_amdgcn_s_sleep(1);
  }
  asm volatile("" ::: "memory");
  return false;
}
// Count this wave once, after all of its earlier LDS operations (LDS serves
// a wave's operations in order).
__device__ __forceinline__ void signal_count(int* c) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(c, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  asm volatile("" ::: "memory");
}

// Max and sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 that hold one
// query row, with the gfx950 lane-swap instructions (no LDS round trip).
// Every lane combines the same two operands in the same order, so all four
// get bitwise-equal results.
__device__ __forceinline__ float row_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float row_sum(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Inclusive prefix sum over the 64 lanes of a wave (all active): shifts
// within each 16-lane row, then row 0's and row 1's last lanes broadcast into
// the rows after them.  DPP moves, no LDS round trip.
__device__ __forceinline__ int wave_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);   // row_bcast:15 into rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);   // row_bcast:31 into rows 2 and 3
  return x;
}

// Two floats rounded (to nearest even) to bf16 and packed, lo in the low
// half: one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}

// The same for f16 (two conversions to nearest even, one pack).
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), f16x2_t));
}

// Probabilities of 8 keys packed into a 16-bit MFMA operand
template <int ELT>
__device__ __forceinline__ u32x4 pack_p(const float (&pr)[8]) {
  if constexpr (ELT == kF16)
    return u32x4{pack_f16x2(pr[0], pr[1]), pack_f16x2(pr[2], pr[3]), pack_f16x2(pr[4], pr[5]),
                 pack_f16x2(pr[6], pr[7])};
  else
    return u32x4{pack_bf16x2(pr[0], pr[1]), pack_bf16x2(pr[2], pr[3]), pack_bf16x2(pr[4], pr[5]),
                 pack_bf16x2(pr[6], pr[7])};
}

// 16x16x32 MFMA on 16-bit operands (8 elements per lane), fp32 accumulation
template <int ELT>
__device__ __forceinline__ f32x4 mfma32(const u32x4& a, const u32x4& b, f32x4 acc) {
  if constexpr (ELT == kF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), acc,
                                                  0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   acc, 0, 0, 0);
}

// Lengths of sequence b, clamped into the documented ranges so that no access
// can leave the buffers even if the caller broke a precondition.  Packed as
// (T << 8) | c with T = l + c < 2^24 (checked on the host) and c <= 128.
__device__ __forceinline__ uint32_t load_seq(const Params& p, int b) {
  int c = p.chunk_lens[b];
  int l = p.ctx_lens[b];
  c = c < 0 ? 0 : (c > p.C_max ? p.C_max : c);
  l = l < 0 ? 0 : l;
  if (l > p.S_max - c) l = p.S_max - c;
  return ((uint32_t)(l + c) << 8) | (uint32_t)c;
}
__device__ __forceinline__ int seq_T(uint32_t s) { return (int)(s >> 8); }
// a value every lane of the wave holds, moved to a scalar register
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ uint32_t uniform(uint32_t x) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)x); }
__device__ __forceinline__ int seq_c(uint32_t s) { return (int)(s & 0xffu); }
template <class C>
__device__ __forceinline__ int seq_tiles(uint32_t s) {
  return seq_c(s) == 0 ? 0 : (seq_T(s) + C::kTileKeys - 1) / C::kTileKeys;
}

// Cost of one tile of a sequence with c chunk tokens: a fixed part for
// streaming the tile, plus one per 16-row block of the unit's c * g query
// rows.  A unit with many rows can take longer on a tile than the tile's
// HBM stream lasts, so workgroups get equal cost rather than equal tiles.
// The weights follow measured tile times (ragged chunks, 1-7 row blocks:
// 2.7, 3.1 and 3.3 us per tile for 1-2, 3-4 and 5-7 blocks).
constexpr int kTileCost = 10;
__device__ __forceinline__ int tile_cost(uint32_t s, int g) { return kTileCost + (seq_c(s) * g + kBlk - 1) / kBlk; }
// Extra costs of a unit: at its start (a first tile that is mostly partial,
// the switch of Q) and at its end (the result's stores and, for units of one
// or two row blocks, the merge of the key-split states; charged after its
// last tile), so ranges that cross more unit boundaries get fewer tiles.  A
// range that starts inside a unit pays for that unit's end.  (Measured: on
// B = 64 with chunks of 5 and 4 query heads per KV head a unit end holds a
// workgroup ~1.6 us and its start ~0.6 us, against ~2.2 us per tile.)
constexpr int kStartSplit = 3, kEndSplit = 9;   // units of one or two row blocks
constexpr int kStartRest = 6, kEndRest = 0;     // larger units
constexpr int kExtraMax = kStartSplit + kEndSplit > kStartRest + kEndRest ? kStartSplit + kEndSplit : kStartRest + kEndRest;
__device__ __forceinline__ bool split_unit(uint32_t s, int g) { return seq_c(s) * g <= 2 * kBlk; }
__device__ __forceinline__ int start_cost(uint32_t s, int g) { return split_unit(s, g) ? kStartSplit : kStartRest; }
__device__ __forceinline__ int end_cost(uint32_t s, int g) { return split_unit(s, g) ? kEndSplit : kEndRest; }
// cost of one unit (one KV head) of a sequence with packed lengths s: its n
// tiles of cost w, its start and its end
__device__ __forceinline__ int unit_cost(int n, int w, uint32_t s, int g) {
  return n > 0 ? n * w + start_cost(s, g) + end_cost(s, g) : 0;
}

// floor(a / b) for 0 <= a < 2^53 and 0 < b < 2^53: the rounded double
// quotient is within one of it, and one exact integer step corrects it
// (much shorter code than a 64-bit integer division).
__device__ __forceinline__ long long div_floor(long long a, long long b) {
  long long q = (long long)((double)a / (double)b);
  const long long r = a - q * b;
  if (r < 0) --q;
  else if (r >= b) ++q;
  return q;
}

// Tile schedule shared by every workgroup of a launch.  The tiles of all
// units form one list [0, N) in (sequence, KV head, tile) order; tile j of
// unit kvh of sequence b starts at cost Hkv cpref[b] + kvh U_b + (j > 0 ?
// S_b + j w_b : 0), w_b its sequence's tile cost, S_b and E_b its unit-start
// and unit-end costs and U_b = n_b w_b + S_b + E_b a unit's cost, out of Wt
// in all.  Range q holds the tiles whose start cost lies in [q Wt / Pe, (q +
// 1) Wt / Pe).  With Pe <= Wt / max_b (w_b + S_b + E_b) no range is empty,
// since consecutive tile starts are at most max_b (w_b + S_b + E_b) apart.
struct Sched {
  int N, Pe, B, Hkv, g;
  bool uni;                 // every tile costs the same and S = 0: the same ranges, found without a search
  long long Wt;
  const uint32_t* seqs;     // packed lengths per sequence
  const int* pref;          // tiles per KV head of the sequences before b
  const int* cpref;         // cost of the units of one KV head of the sequences before b
  // range of tile j of unit kvh of sequence b (n tiles per unit)
  __device__ int owner(int b, int kvh, int j, int n) const {
    if (uni) return (int)div_floor((long long)(Hkv * pref[b] + kvh * n + j) * Pe, N);
    const int w = tile_cost(seqs[b], g);
    const long long c =
        (long long)Hkv * cpref[b] + (long long)kvh * unit_cost(n, w, seqs[b], g) + (j > 0 ? start_cost(seqs[b], g) + j * w : 0);
    return (int)div_floor(c * Pe, Wt);
  }
  // first tile of range q (N for q = Pe); every lane of the wave takes part
  __device__ int range_begin(int q) const {
    if (q >= Pe) return N;
    if (uni) return (int)div_floor((long long)q * N + Pe - 1, Pe);
    const long long X = (long long)q * Wt;
    // the last sequence b with Hkv cpref[b] Pe <= X: a 64-ary search of the
    // B + 1 prefix entries; that sequence has tiles, as Hkv cpref[b + 1] Pe > X
    const int lane = threadIdx.x & 63;
    const int step = (B + 64) / 64;
    const int i1 = min(lane * step, B);
    const long long hp = (long long)Hkv * Pe;
    const unsigned long long m1 = __ballot(cpref[i1] * hp <= X);
    const int base = (63 - __builtin_clzll(m1)) * step;
    const int i2 = min(base + lane, B);
    const unsigned long long m2 = __ballot(lane < step && cpref[i2] * hp <= X);
    const int b = __builtin_amdgcn_readfirstlane(base + 63 - __builtin_clzll(m2));
    const int n = pref[b + 1] - pref[b];   // tiles per unit of sequence b
    const int w = tile_cost(seqs[b], g);
    // the unit of sequence b whose cost interval holds X, then the first of
    // its tiles that starts at or after X (or the next unit's first tile)
    const long long rem = X - cpref[b] * hp;   // >= 0
    const long long U = (long long)unit_cost(n, w, seqs[b], g) * Pe;
    const int kvh = (int)div_floor(rem, U);
    const long long rem2 = rem - kvh * U;
    int j = 0;
    if (rem2 > 0) {
      const long long den = (long long)w * Pe;
      j = (int)div_floor(rem2 - (long long)start_cost(seqs[b], g) * Pe + den - 1, den);
      j = j < 1 ? 1 : j > n ? n : j;   // n: the next unit's first tile
    }
    return Hkv * pref[b] + kvh * n + j;
  }
};

// Position of a tile: sequence, KV head, tile index inside the unit, and the
// sequence's packed lengths.
struct Cursor {
  int b, kvh, j;
  uint32_t s;
};

// Merge every piece of up to two units: those that this workgroup merges
// through the workspace, run by its consumer threads after its own tiles.  A
// unit's pieces come from ranges qf..ql; range q's piece is its first
// segment (slot 2q), except for range qf when it starts before the unit:
// then it is qf's last segment (slot_first = 2 qf + 1).  The (row, 4 d)
// items of both units form one list, and each thread takes three items per
// round and issues all their loads before it waits, so the two units' loads
// go out together.  Unit u is described by e_u = {unit, qf, ql, slot_first}.
template <int D, bool NT>
__device__ __forceinline__ void merge_units(const Params& p, const uint32_t* seqs, int ctid, const int* e_a,
                                         const int* e_b, bool has_a, bool has_b) {
  const __amdgpu_buffer_rsrc_t ws_o_rsrc = __builtin_amdgcn_make_buffer_rsrc(p.ws_o, 0, p.ws_o_bytes, kBufferFormat);
  const __amdgpu_buffer_rsrc_t ws_lse_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(p.ws_lse, 0, p.ws_lse_bytes, kBufferFormat);
  const int g = p.g;
  int ua = 0, qfa = 0, qla = -1, sfa = 0, ub = 0, qfb = 0, qlb = -1, sfb = 0;
  if (has_a) {
    ua = uniform(e_a[0]);
    qfa = uniform(e_a[1]);
    qla = uniform(e_a[2]);
    sfa = uniform(e_a[3]);
  }
  if (has_b) {
    ub = uniform(e_b[0]);
    qfb = uniform(e_b[1]);
    qlb = uniform(e_b[2]);
    sfb = uniform(e_b[3]);
  }
  const int n_a = has_a ? seq_c(uniform(seqs[ua / p.Hkv])) * g * (D / 4) : 0;
  const int n_b = has_b ? seq_c(uniform(seqs[ub / p.Hkv])) * g * (D / 4) : 0;
  const int n_items = n_a + n_b;
  const int np_max = max(qla - qfa, qlb - qfb) + 1;   // pieces of the larger unit
  constexpr int kBatch = 4;   // pieces loaded per item before combining
  constexpr int kItems = 3;   // items per thread and round
  for (int base = ctid; base < n_items; base += kItems * kCThreads) {
    float m[kItems], z[kItems];
    f32x4 acc[kItems];
    int srow0[kItems], qf[kItems], ql[kItems], sf[kItems], d0[kItems];
    size_t orow[kItems];
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
      m[it] = -INFINITY;
      z[it] = 0.f;
      acc[it] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int idx = base + it * kCThreads;
      const bool in_a = idx < n_a;
      const int unit = in_a ? ua : ub;
      const int local = in_a ? idx : idx - n_a;
      const int r = local / (D / 4);
      d0[it] = 4 * (local - r * (D / 4));
      qf[it] = in_a ? qfa : qfb;
      ql[it] = idx < n_items ? (in_a ? qla : qlb) : -1;   // no pieces for a lane past the items
      sf[it] = in_a ? sfa : sfb;
      srow0[it] = r;
      const int b = unit / p.Hkv;
      orow[it] = (size_t)(b * p.C_max + r / g) * p.Hq + (unit - b * p.Hkv) * g + r % g;
    }
    for (int k0 = 0; k0 < np_max; k0 += kBatch) {
      float lq[kItems][kBatch];
      f32x4 x[kItems][kBatch];
#pragma unroll
      for (int it = 0; it < kItems; ++it) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int q = qf[it] + k0 + u;
          const int srow = (k0 + u == 0 ? sf[it] : 2 * q) * p.Rcap + srow0[it];
          if (q <= ql[it]) {
            lq[it][u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ws_lse_rsrc, srow * 4, 0,
                                                                                     kDeviceCoherent));
            x[it][u] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                     ws_o_rsrc, (srow * D + d0[it]) * 4, 0, kDeviceCoherent));
          }
        }
      }
#pragma unroll
      for (int it = 0; it < kItems; ++it) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          if (qf[it] + k0 + u > ql[it]) break;
          if (lq[it][u] == -INFINITY) continue;   // a piece in which this row sees no key
          const float nm = fmaxf(m[it], lq[it][u]);
          const float a = expf(m[it] - nm);
          const float w = expf(lq[it][u] - nm);
          z[it] = z[it] * a + w;
          acc[it] = acc[it] * a + w * x[it][u];
          m[it] = nm;
        }
      }
    }
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
      if (base + it * kCThreads >= n_items) continue;
      // (z = 0: a row that sees no key in any piece)
      const f32x4 res = acc[it] * (z[it] > 0.f ? 1.f / z[it] : 0.f);
      const float res_lse = z[it] > 0.f ? m[it] + logf(z[it]) : -INFINITY;
      if constexpr (NT) {
        __builtin_nontemporal_store(res, reinterpret_cast<f32x4*>(p.out + orow[it] * D + d0[it]));
        if (d0[it] == 0) __builtin_nontemporal_store(res_lse, p.lse + orow[it]);
      } else {
        *reinterpret_cast<f32x4*>(p.out + orow[it] * D + d0[it]) = res;
        if (d0[it] == 0) p.lse[orow[it]] = res_lse;
      }
    }
  }
  if (ctid == 0) {   // ready for the next call
    if (has_a) __hip_atomic_store(p.counters + ua, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (has_b) __hip_atomic_store(p.counters + ub, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// TREE: the draft region obeys per-token draft-mask words instead of the
// chain mask.  PAGED: the KV cache is a pool of pages found through a block
// table.  MODE kModeHold (launches whose units have at most two 16-row
// blocks): the piece of a range's first segment is held in LDS until three
// quarters into the range.  MODE kModeNt: results are stored with the
// non-temporal policy (launches with many units per workgroup and a large
// output).
template <int ELT, int D, bool TREE, bool PAGED, int MODE>
__global__ __launch_bounds__(kThreads, 1) void verify_attn_kernel(Params p) {
  constexpr bool HOLD = MODE == kModeHold;
  constexpr bool NT = MODE == kModeNt;
  constexpr bool W16 = ELT != kF32;   // 16-bit elements
  using C = Cfg<W16, D>;
  __shared__ __attribute__((aligned(16))) char smem[kStages * C::kStage];
  __shared__ uint32_t seqs[kMaxSeqs];     // packed (T, c) of every sequence of the launch
  __shared__ int pref[kMaxSeqs + 1];      // tiles per KV head of the sequences before b
  // the cost of one KV head's tiles of the sequences before b; with HOLD it
  // shares its LDS with the held piece (O rows, then the rows' max and sum),
  // which is written only once the schedule has been made
  __shared__ __attribute__((aligned(16))) char piece_lds[HOLD ? C::kPieceLds : 16];
  __shared__ int cpref_own[HOLD ? 1 : kMaxSeqs + 1];
  int* const cpref = HOLD ? reinterpret_cast<int*>(piece_lds) : cpref_own;
  __shared__ float mst[kConsumers][2][kBlk];   // key-split merge: max and sum of each wave's rows
  __shared__ int sh_flag[2];              // "this piece completed its unit", for the two pieces
  __shared__ int sh_direct;               // the next range's piece of the last unit had arrived at the last tile
  __shared__ int sh_share[2][4];          // unit, qf, ql, slot_first of the units of tiles g0 and g1 - 1
  __shared__ int full_cnt[kStages];       // producer waves whose loads of the stage's tile have landed
  __shared__ int empty_cnt[kStages];      // consumer waves done with the stage's tile
  __shared__ int cb_cnt;                  // consumer waves that reached a consumer barrier
  __shared__ int pub_arrive[2];           // consumer waves whose stores of piece k have completed

  const int pid = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const bool producer = wave < kProducers;
  const int wc = wave - kProducers;       // consumer wave index
  const int ctid = tid - 64 * kProducers; // consumer thread index
  const int lm = lane & 15;               // row (or key, or d) inside a 16-wide MFMA block
  const int lg = lane >> 4;               // which quarter of the MFMA k dimension this lane feeds
  const int B = p.B, Hkv = p.Hkv, g = p.g;
  // set when one of this wave's hand-off waits gave up; raised once in the
  // workspace's sticky status word when the wave ends
  bool gave_up = false;
  auto report_give_up = [&](bool gave) {
    if (gave && lane == 0) __hip_atomic_fetch_or(p.status, kGaveUp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };

  // ---- padding rows c_b <= i < C_max of the sequences b = pid (mod P):
  // out = 0, lse = -inf; written by threads t0, t0 + stride, ..., with the
  // non-temporal policy (nothing reads them back).  Written at the start,
  // while the first tiles stream in, they cost the ragged-chunk workload
  // (13.5 MB of padding rows) 2.2 us more than from the producers at the end.
  auto pad_rows = [&](int t0, int stride) {
    for (int b = pid; b < B; b += p.P) {
      const int c = seq_c(seqs[b]);
      const int pad_rows_b = (p.C_max - c) * p.Hq;
      for (int idx = t0; idx < pad_rows_b * (D / 4); idx += stride) {
        const int r = idx / (D / 4);
        const int d4 = idx - r * (D / 4);
        const int i = c + r / p.Hq;
        const int h = r % p.Hq;
        const size_t orow = (size_t)(b * p.C_max + i) * p.Hq + h;
        __builtin_nontemporal_store(f32x4{0.f, 0.f, 0.f, 0.f}, reinterpret_cast<f32x4*>(p.out + orow * D + 4 * d4));
        if (d4 == 0) __builtin_nontemporal_store(-INFINITY, p.lse + orow);
      }
    }
  };

  // Cursor of global tile t: a 64-ary search of the prefix sums, done by a
  // whole wave (two LDS reads and two ballots).
  auto locate = [&](int t) {
    const int tq = t / Hkv;                      // tiles per KV head before t's sequence, at most
    const int step = (B + 64) / 64;              // B + 1 prefix entries in 64 groups
    const int i1 = min(lane * step, B);
    const unsigned long long m1 = __ballot(pref[i1] <= tq);
    const int base = (63 - __builtin_clzll(m1)) * step;
    const int i2 = min(base + lane, B);
    const unsigned long long m2 = __ballot(lane < step && pref[i2] <= tq);
    Cursor cu;
    cu.b = uniform(base + 63 - __builtin_clzll(m2));
    cu.s = uniform(seqs[cu.b]);
    const int n = seq_tiles<C>(cu.s);
    const int off = t - Hkv * uniform(pref[cu.b]);
    cu.kvh = off / n;
    cu.j = off - cu.kvh * n;
    return cu;
  };
  Sched sc;
  sc.B = B;
  sc.Hkv = Hkv;
  sc.g = g;
  sc.seqs = seqs;
  sc.pref = pref;
  sc.cpref = cpref;
  // every tile costs at most w_hi, so with at most Wt / w_hi ranges (and at
  // least one when there are tiles) no range is empty
  const int w_hi = kTileCost + (p.C_max * g + kBlk - 1) / kBlk + kExtraMax;
  auto set_totals = [&](int tiles_per_head, int cost_per_head) {
    sc.N = tiles_per_head * Hkv;   // tiles of all units (< 2^30, host check)
    sc.Wt = (long long)Hkv * cost_per_head;
    long long pe = div_floor(sc.Wt, w_hi);
    if (pe < 1) pe = sc.N > 0 ? 1 : 0;
    sc.Pe = pe < p.P ? (int)pe : p.P;
    sc.uni = kExtraMax == 0 && sc.Wt == (long long)sc.N * w_hi;
  };

  // ---- prologue, by wave 0 alone while the other waves wait at one
  // barrier (every wave doing it was issue-bound): the lengths, tile and cost
  // prefix sums into LDS, then this workgroup's range [g0, g1) and its first
  // tile.  Lane l owns the contiguous sequences [l per, (l + 1) per).  Every
  // range is streamed in order.
  __shared__ int sh_sched[12];
  if (wave == 0) {
    const int per = (B + 63) / 64;
    const int b_lo = min(lane * per, B);
    const int b_hi = min(b_lo + per, B);
    int my_tiles = 0, my_cost = 0;   // sums < 2^31 (host check)
    uint32_t my_s = 0;               // (B <= 64) the packed lengths of sequence lane
    for (int b = b_lo; b < b_hi; ++b) {
      const uint32_t s = load_seq(p, b);
      seqs[b] = s;
      my_s = s;
      my_tiles += seq_tiles<C>(s);
      my_cost += unit_cost(seq_tiles<C>(s), tile_cost(s, g), s, g);
    }
    const int incl = wave_scan(my_tiles), cincl = wave_scan(my_cost);
    const int total = __builtin_amdgcn_readlane(incl, 63);
    const int ctotal = __builtin_amdgcn_readlane(cincl, 63);
    // exclusive prefixes: pref[b_lo] and cpref[b_lo] (the totals in lanes
    // without sequences)
    const int ex = incl - my_tiles, cex = cincl - my_cost;
    int run = ex, crun = cex;
    for (int b = b_lo; b < b_hi; ++b) {
      pref[b] = run;
      cpref[b] = crun;
      run += seq_tiles<C>(seqs[b]);
      crun += unit_cost(seq_tiles<C>(seqs[b]), tile_cost(seqs[b], g), seqs[b], g);
    }
    if (lane == 63) {
      pref[B] = total;
      cpref[B] = ctotal;
    }
    if (lane < kStages) {
      full_cnt[lane] = 0;
      empty_cnt[lane] = 0;
    }
    if (lane == 0) cb_cnt = 0;
    if (lane < 2) {
      pub_arrive[lane] = 0;
      sh_flag[lane] = 0;
    }
    set_totals(total, ctotal);
    // With at most 64 sequences lane l holds sequence l (one per lane), and
    // with ex = pref[min(l, B)], cex = cpref[min(l, B)] the searches below
    // run on registers and ballots instead of LDS round trips: the same
    // results as Sched::range_begin and locate.
    const bool in_regs = B <= 64;
    auto range_begin_w0 = [&](int q) {
      if (!in_regs || q >= sc.Pe || sc.uni) return sc.range_begin(q);
      const long long X = (long long)q * sc.Wt, hp = (long long)Hkv * sc.Pe;
      // lane 0 (cex = 0) always passes, lanes from B on (cex = ctotal, and
      // ctotal hp = Pe Wt > X) never do
      const unsigned long long m = __ballot((long long)cex * hp <= X);
      const int b = 63 - __builtin_clzll(m);
      const int n = __builtin_amdgcn_readlane(my_tiles, b);
      const uint32_t s_b = (uint32_t)__builtin_amdgcn_readlane((int)my_s, b);
      const int w = tile_cost(s_b, g);
      const long long rem = X - (long long)__builtin_amdgcn_readlane(cex, b) * hp;
      const long long U = (long long)unit_cost(n, w, s_b, g) * sc.Pe;
      const int kvh = (int)div_floor(rem, U);
      const long long rem2 = rem - kvh * U;
      int j = 0;
      if (rem2 > 0) {
        const long long den = (long long)w * sc.Pe;
        j = (int)div_floor(rem2 - (long long)start_cost(s_b, g) * sc.Pe + den - 1, den);
        j = j < 1 ? 1 : j > n ? n : j;
      }
      return Hkv * __builtin_amdgcn_readlane(ex, b) + kvh * n + j;
    };
    auto locate_w0 = [&](int t) {
      if (!in_regs) return locate(t);
      // lane 0 (ex = 0) always passes, lanes from B on (ex = total > t / Hkv
      // for t < N) never do
      const unsigned long long m = __ballot(ex <= t / Hkv);
      const int b = 63 - __builtin_clzll(m);
      Cursor cu;
      cu.b = b;
      cu.s = (uint32_t)__builtin_amdgcn_readlane((int)my_s, b);
      const int n = seq_tiles<C>(cu.s);
      const int off = t - Hkv * __builtin_amdgcn_readlane(ex, b);
      cu.kvh = off / n;
      cu.j = off - cu.kvh * n;
      return cu;
    };
    int g0 = 0, g1 = 0;
    Cursor first = {0, 0, 0, 0u};
    if (pid < sc.Pe) {
      g0 = range_begin_w0(pid);
      g1 = range_begin_w0(pid + 1);
      first = locate_w0(g0);
    }
    if (lane == 0) {
      sh_sched[0] = total;
      sh_sched[1] = ctotal;
      sh_sched[9] = sc.Pe;
      sh_sched[10] = sc.uni ? 1 : 0;
      sh_sched[2] = g0;
      sh_sched[3] = g1;
      sh_sched[6] = first.b;
      sh_sched[7] = first.kvh;
      sh_sched[8] = first.j;
    }
  }
  __syncthreads();
  if (wave != 0) {
    sc.N = uniform(sh_sched[0]) * Hkv;
    sc.Wt = (long long)Hkv * uniform(sh_sched[1]);
    sc.Pe = uniform(sh_sched[9]);
    sc.uni = uniform(sh_sched[10]) != 0;
  }
  if (pid >= sc.Pe) {
    pad_rows(tid, kThreads);
    return;
  }
  const int g0 = uniform(sh_sched[2]);
  const int g1 = uniform(sh_sched[3]);
  const int count = g1 - g0;
  Cursor first;
  first.b = uniform(sh_sched[6]);
  first.kvh = uniform(sh_sched[7]);
  first.j = uniform(sh_sched[8]);
  first.s = uniform(seqs[first.b]);
  // the first tile of unit (b, kvh) after cursor cu's unit
  auto next_unit = [&](Cursor& cu) {
    cu.j = 0;
    if (++cu.kvh == Hkv) {
      cu.kvh = 0;
      do {
        ++cu.b;
      } while (seq_tiles<C>(uniform(seqs[cu.b])) == 0);   // in range: the next tile exists
      cu.s = uniform(seqs[cu.b]);
    }
  };
  // the tile after cursor cu
  auto advance = [&](Cursor& cu) {
    if (++cu.j == seq_tiles<C>(cu.s)) next_unit(cu);
  };
  // the first tile of the segment after the one cu is in (cu at position v
  // of the range): its position v_next and cursor
  auto next_segment = [&](const Cursor& cu, int v, int& v_next) {
    v_next = min(v + seq_tiles<C>(cu.s) - cu.j, count);
    Cursor nx = cu;
    if (v_next < count) next_unit(nx);
    return nx;
  };

  // ---- producers: K/V tile of cursor cu straight from HBM into stage st.
  // Each 64-lane load fills 64 consecutive 16-byte LDS slots (1 KB of
  // consecutive cache rows with their pad slots); a pad lane re-reads a chunk
  // of its own row, and within a partial tile the lanes past its last row
  // re-read that row.  K loads that would start past the last row are not
  // issued: those slots keep whatever an earlier tile or merge left there,
  // and the consumers mask the keys.  A masked key has probability 0 but
  // must meet finite V values: the first tile of each stage loads every V
  // slot (LDS starts undefined), later tiles skip the V loads past the last
  // row too, whose slots then hold rows of an earlier tile (the key-split
  // merge's scratch stays in the K half).  Paged caches load every V slot
  // (skipping measured slower there: 77.2 -> 79.5 us on B = 64 with 16-token
  // pages, against 68.2 -> 67.2 us with a contiguous cache).  The two waves of a producer pair
  // issue the K and V instructions of even and odd index.
  const int pw = wave & 1;
  // (paged) the pool pages of the tile of cu, one per lane of a producer
  // wave: lane l holds the page of the tile's l-th page (at most 33 of them:
  // pages hold at least 8 tokens, tiles at most 256).  Out-of-range table
  // entries are clamped into the pool.
  auto load_pages = [&](const Cursor& cu) {
    int r = 0;
    if constexpr (PAGED) {
      const int T = seq_T(cu.s);
      const int hi = T - (seq_tiles<C>(cu.s) - 1 - cu.j) * C::kTileKeys;
      const int lo = hi > C::kTileKeys ? hi - C::kTileKeys : 0;
      const int fp = lo >> p.page_shift;
      if (lane <= ((hi - 1) >> p.page_shift) - fp)
        r = min(max(p.block_table[(size_t)cu.b * p.pages_per_seq + fp + lane], 0), p.num_pages - 1);
    }
    return r;
  };
  auto dma = [&](const Cursor& cu, int st, int pg, bool all_v) {
    const int T = seq_T(cu.s);
    const int hi = T - (seq_tiles<C>(cu.s) - 1 - cu.j) * C::kTileKeys;
    const int lo = hi > C::kTileKeys ? hi - C::kTileKeys : 0;
    const int last = hi - lo - 1;
    // K/V slab of the unit; byte offsets inside it fit in 32 bits (host check)
    const size_t slab = ((size_t)cu.b * Hkv + cu.kvh) * (size_t)p.S_max * C::kRowBytes;
    const char* kp = p.k + slab + (size_t)lo * C::kRowBytes;
    const char* vp = p.v + slab + (size_t)lo * C::kRowBytes;
    char* kl = smem + st * C::kStage;
    char* vl = kl + C::kLdsK;
#pragma unroll
    for (int k = 0; k < kMaxDma; ++k) {
      const int i = pw + 2 * k;
      const int sl = 64 * i + lane;
      // source offset of LDS slot sl in each half (a pad slot re-reads its
      // row's last chunk)
      const int krow_ = sl / C::kSlotsK;
      const uint32_t koff =
          (uint32_t)min(krow_, last) * C::kRowBytes + 16u * min(sl - krow_ * C::kSlotsK, C::kChunks - 1);
      const int vrow_ = sl / C::kSlotsV;
      const uint32_t voff =
          (uint32_t)min(vrow_, last) * C::kRowBytes + 16u * min(sl - vrow_ * C::kSlotsV, C::kChunks - 1);
      const char* ksrc = kp + koff;
      const char* vsrc = vp + voff;
      if constexpr (PAGED) {
        // row j of the sequence: page table[j >> shift] of the pool, row
        // j & (page - 1) of the unit's KV head in it
        const int sh = p.page_shift;
        const int fp = lo >> sh;
        const size_t page_bytes = ((size_t)Hkv << sh) * C::kRowBytes;
        const size_t head_bytes = ((size_t)cu.kvh << sh) * C::kRowBytes;
        const int kj = lo + min(krow_, last), vj = lo + min(vrow_, last);
        const int kpage = __shfl(pg, (kj >> sh) - fp), vpage = __shfl(pg, (vj >> sh) - fp);
        ksrc = p.k + (size_t)kpage * page_bytes + head_bytes + (size_t)(kj & ((1 << sh) - 1)) * C::kRowBytes +
               16u * min(sl - krow_ * C::kSlotsK, C::kChunks - 1);
        vsrc = p.v + (size_t)vpage * page_bytes + head_bytes + (size_t)(vj & ((1 << sh) - 1)) * C::kRowBytes +
               16u * min(sl - vrow_ * C::kSlotsV, C::kChunks - 1);
      }
      // a K load whose first row is past the tile's keys is skipped: those
      // scores are masked whatever the slots hold
      if (i < C::kInstK && sl < C::kTileKeys * C::kSlotsK && (64 * i) / C::kSlotsK <= last)
        __builtin_amdgcn_global_load_lds(ksrc, (__attribute__((address_space(3))) void*)(kl + 1024 * i), 16, 0,
                                         kStreaming);
      if (i < C::kInstV && sl < C::kTileKeys * C::kSlotsV && (PAGED || all_v || (64 * i) / C::kSlotsV <= last))
        __builtin_amdgcn_global_load_lds(vsrc, (__attribute__((address_space(3))) void*)(vl + 1024 * i), 16, 0,
                                         kStreaming);
    }
  };


  // ---- consumer roles for the unit of cursor cu.  Rows are cut into
  // n_rb 16-row blocks; consumer wave wc takes row block rb = wc % n_rbp, and
  // the nks waves of a row block (its key slots) share every tile's key
  // blocks: wave kslot takes the pairs (kb, kb + nks) for kb = kslot,
  // kslot + 2 nks, ...  (nks <= kNKB / 2, so every wave has whole pairs).
  // One row block: four waves (nks = 4).  Two: two waves per block (the
  // merge of the waves' partial states at every unit end costs more than the
  // compute that two more waves per block would take over), four waves idle.
  // From three blocks on (n_rbp = 8), a wave computes its block's whole
  // tile, which is cheaper than merging at the end of every unit.
  int R = 0, n_rbp = 1, nks = 1, rb = 0, kslot = 0, l_ctx = 0, row = 0, tok = 0, vis = 0;
  bool active = false, row_valid = false;
  uint64_t tmask = 0;   // (tree drafts) this lane's row: bit k = sees draft key l_ctx + k
  // (tree drafts) the row's mask word of the current segment's unit and of
  // the next segment's, loaded with that segment's Q: a load issued at the
  // unit's start would be waited for inside the pair loop, and that wait
  // would cover the Q prefetch and the stores issued before it
  uint64_t tm_r = 0, tm_n = 0;
  // x / g for a row 0 <= x < 128 of a unit, by a float reciprocal: exact
  // there, as (x + 1/2) / g lies at least 1 / (2 g) from an integer
  const float inv_g = 1.f / (float)g;
  auto div_g = [&](int x) { return (int)(((float)x + 0.5f) * inv_g); };
  auto rbp_shift = [&](int n_rb) { return n_rb <= 1 ? 0 : n_rb <= 2 ? 1 : 3; };   // log2 n_rbp
  // waves that share a row block's tiles (key slots)
  auto key_slots = [&](int n_rb, int sh) { return n_rb == 2 ? 2 : min(kConsumers >> sh, C::kNKB / 2); };
  auto roles = [&](const Cursor& cu) {
    const int c = seq_c(cu.s);
    R = c * g;
    l_ctx = seq_T(cu.s) - c;
    const int n_rb = (R + kBlk - 1) / kBlk;
    const int sh = rbp_shift(n_rb);
    n_rbp = 1 << sh;
    nks = key_slots(n_rb, sh);
    rb = producer ? 0 : wc & (n_rbp - 1);
    kslot = producer ? nks : wc >> sh;
    active = !producer && rb < n_rb && kslot < nks;
    row = rb * kBlk + lm;
    row_valid = active && row < R;
    tok = row_valid ? div_g(row) : 0;
    if constexpr (TREE) {
      // every key below the sequence end passes the compare; the draft
      // keys are then filtered by the row's word
      vis = 0x7fffffff;
      tmask = tm_r;   // 0 for rows that are not valid
    } else {
      vis = row_valid ? l_ctx + tok : 0x7fffffff;   // last visible key of this lane's row
    }
  };
  // Q chunks of this lane's row for the unit of cu (zero for invalid rows):
  // chunk 4J + lg of the row feeds the J-th score MFMA.  Consumers only.
  auto load_q = [&](const Cursor& cu, u32x4* dst, uint64_t& mdst) {
    const int c = seq_c(cu.s);
    const int uR = c * g;
    const int n_rb = (uR + kBlk - 1) / kBlk;
    const int sh = rbp_shift(n_rb);
    const int rb_ = wc & ((1 << sh) - 1);
    const int ks_ = wc >> sh;
    const int row_ = rb_ * kBlk + lm;
    const bool ok = rb_ < n_rb && ks_ < key_slots(n_rb, sh) && row_ < uR;
    const int tk = ok ? div_g(row_) : 0;
    const char* qrow =
        p.q + ((size_t)(cu.b * p.C_max + tk) * p.Hq + cu.kvh * g + (ok ? row_ - tk * g : 0)) * C::kRowBytes;
#pragma unroll
    for (int J = 0; J < C::kQJ; ++J)
      dst[J] = ok ? *reinterpret_cast<const u32x4*>(qrow + 16 * (4 * J + lg)) : u32x4{0u, 0u, 0u, 0u};
    if constexpr (TREE) mdst = ok ? p.draft_mask[cu.b * p.C_max + tk] : 0;
  };

  // Publication of pieces (at most two per workgroup: its first and last
  // segment).  Two tiles after a piece's stores, each consumer wave waits for
  // its own stores (a wait no tile load shares) and arrives on an LDS
  // counter; the last of the eight counts the piece on its unit's arrival
  // counter.  The counts are read back after the loop, where the unit's
  // merge is decided.  The loop runs idle iterations after the last tile
  // until every piece is counted.  The last segment's piece of a unit that
  // starts in the range is not published in the loop: it stays in registers
  // (pend_direct) for the merge after the loop.
  struct Pub {
    int state;   // 0 stored, 1 counted, 2 no piece, 3 held in LDS
    int unit, v, rows;
  };

  // ---- consumers.  Per-segment state of a lane: O^T blocks, running max
  // (log2 units, the same in the four lanes of a row), this lane's share of
  // the row sum, and the Q operand of this unit and of the next.
  f32x4 o[C::kDB];
#pragma unroll
  for (int db = 0; db < C::kDB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  u32x4 qr[C::kQJ], qn[C::kQJ];
#pragma unroll
  for (int J = 0; J < C::kQJ; ++J) qn[J] = u32x4{0u, 0u, 0u, 0u};
  float m_run = -INFINITY, l_lane = 0.f;
  Pub pub0 = {2, 0, 0, 0}, pub1 = {2, 0, 0, 0};
  int n_pub = 0;
  // The consumer wave that counts piece k on its unit's arrival counter sets
  // bit k of counted and keeps the counter's previous value in cnt[k] (lane
  // 0); with HOLD the last piece to arrive merges the unit after the loop.
  // (Reading the counter back after the loop instead costs one more round
  // trip at the end of the range, which measured slower there.)
  int counted = 0;
  int cnt[2] = {0, 0};
  int ncb = 0;   // consumer barriers passed
  auto cbar = [&]() {
    ++ncb;
    signal_count(&cb_cnt);
    gave_up |= !wait_count(&cb_cnt, kConsumers * ncb, p.spin_limit);
  };

  // The first unit's Q arrives through qn, so that qr is only ever written
  // from registers and the score MFMAs never wait for a load.  The producers
  // start at once: the Q loads need not go out before the first tile's.
  if (!producer) load_q(first, qn, tm_n);
  if (producer) {
    // Producer pair grp streams the tiles v = grp, grp + 2, ... of the
    // workgroup's order into stage grp: it waits until all consumers have
    // released the stage's previous tile, issues the loads, waits for its own
    // loads to land and counts itself on the stage's fill counter.  The two
    // pairs run independently, so one tile's loads are issued while the
    // other's are still in flight; only tile 1 waits until tile 0 has landed,
    // so that at the start, when every workgroup asks for its first tiles at
    // once, tile 0 is not delivered interleaved with tile 1.
    const int grp = wave >> 1;
    Cursor cu = first;
    int v = grp;
    if (grp == 1 && count > 1) advance(cu);
    int pg = 0;   // (paged) the pages of the pair's next tile
    if constexpr (PAGED)
      if (v < count) pg = load_pages(cu);
    for (; v < count; v += 2) {
      if (v >= 2) gave_up |= !wait_count(&empty_cnt[grp], kConsumers * (v >> 1), p.spin_limit);
      if (v == 1) gave_up |= !wait_count(&full_cnt[0], 2, p.spin_limit);
      dma(cu, grp, pg, v < 2);
      if constexpr (PAGED) {
        // the next tile's table entries ride the wait for this tile's loads
        if (v + 2 < count) {
          advance(cu);
          advance(cu);
          pg = load_pages(cu);
        }
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      signal_count(&full_cnt[grp]);
      if constexpr (!PAGED) {
        if (v + 2 < count) {
          advance(cu);
          advance(cu);
        }
      }
    }
    // the padding rows of the workgroup's sequences, by the producers once
    // their tiles are in, while the consumers compute the last ones
    pad_rows(tid, kProducers * 64);
    report_give_up(gave_up);
    return;
  }
  // Only the units of the range's first and last tile can be shared with
  // other workgroups.  Their piece bookkeeping (the ranges qf..ql that hold
  // their tiles, and the slot of range qf's piece) is worked out now, while
  // the first tile streams in, rather than at the end.
  if (wc == 0) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int t = k == 0 ? g0 : g1 - 1;
      const Cursor cu = locate(t);
      const int n = seq_tiles<C>(cu.s);
      const int qf = sc.owner(cu.b, cu.kvh, 0, n);
      const int ql = sc.owner(cu.b, cu.kvh, n - 1, n);
      const int slot_first = 2 * qf + (sc.range_begin(qf) < t - cu.j ? 1 : 0);   // whole wave: a ballot search
      if (lane == 0) {
        sh_share[k][0] = cu.b * Hkv + cu.kvh;
        sh_share[k][1] = qf;
        sh_share[k][2] = ql;
        sh_share[k][3] = slot_first;
      }
    }
  }
#pragma unroll
  for (int J = 0; J < C::kQJ; ++J) qr[J] = qn[J];
#pragma unroll
  for (int J = 0; J < C::kQJ; ++J) asm volatile("" : "+v"(qr[J])::"memory");
  if constexpr (TREE) {
    tm_r = tm_n;
    asm volatile("" : "+v"(tm_r)::"memory");
  }
  {
    int v1;
    const Cursor c1 = next_segment(first, 0, v1);
    if (v1 < count) load_q(c1, qn, tm_n);   // the second segment's Q
  }
  Cursor cur = first;                  // cursor of the tile being computed
  int seg_g = g0;
  // results of the segment that ended in the previous iteration, stored at
  // the top of this one: o[] (this wave's d blocks), and per lane the output
  // (or workspace) row, 1 / row sum and the row's lse
  bool pend = false, pend_whole = false, pend_ok = false;
  int pend_row = 0;
  float pend_inv = 0.f, pend_lse = 0.f;
  // When the range's last segment starts a unit that continues into later
  // ranges, its piece stays in registers (pend_direct) and, if the unit has
  // just one more piece (the next range's first segment) and that piece has
  // arrived (the unit's counter, read at the last tile into probe by wave 0,
  // lane 0), is merged with it after the loop into the final rows; else it
  // is stored and counted then, as the loop would have.
  bool pend_direct = false;
  int pend_k = 0, probe = 0;

  for (int v = 0;; ++v) {
    // (a held piece is stored by iteration count - 1, so no piece is held here)
    if (v >= count && pub0.state != 0 && pub1.state != 0 && !pend) break;
    if (pend && pend_ok && !pend_direct) {
      const int s_db = nks <= C::kDB ? C::kDB / nks : 1;
      const int d_lo = kslot * s_db, d_hi = d_lo + s_db;   // this wave's d blocks
      if (pend_whole) {
        float* dst = p.out + (size_t)pend_row * D;
        if (kslot == 0 && lg == 0) {
          if constexpr (NT) __builtin_nontemporal_store(pend_lse, p.lse + pend_row);
          else p.lse[pend_row] = pend_lse;
        }
#pragma unroll
        for (int db = 0; db < C::kDB; ++db)
          if (db >= d_lo && db < d_hi) {
            if constexpr (NT)
              __builtin_nontemporal_store(o[db] * pend_inv, reinterpret_cast<f32x4*>(dst + 16 * db + 4 * lg));
            else
              *reinterpret_cast<f32x4*>(dst + 16 * db + 4 * lg) = o[db] * pend_inv;
          }
      } else {
        // read by another workgroup, possibly on another XCD
        const __amdgpu_buffer_rsrc_t ws_o_rsrc =
            __builtin_amdgcn_make_buffer_rsrc(p.ws_o, 0, p.ws_o_bytes, kBufferFormat);
        const __amdgpu_buffer_rsrc_t ws_lse_rsrc =
            __builtin_amdgcn_make_buffer_rsrc(p.ws_lse, 0, p.ws_lse_bytes, kBufferFormat);
        if (kslot == 0 && lg == 0)
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, pend_lse), ws_lse_rsrc, pend_row * 4, 0,
                                                kDeviceCoherent);
#pragma unroll
        for (int db = 0; db < C::kDB; ++db)
          if (db >= d_lo && db < d_hi)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, o[db] * pend_inv), ws_o_rsrc,
                                                   (pend_row * D + 16 * db + 4 * lg) * 4, 0, kDeviceCoherent);
      }
    }
    if (pend && !pend_direct) {
      // the next tile starts a new segment
#pragma unroll
      for (int db = 0; db < C::kDB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    pend = false;
    if (HOLD && pub0.state == 3 && v == pub0.v) {
      // the held piece (the first segment's, slot 2 pid) goes out now, while
      // the range's last tile streams in; it is counted two iterations later
      cbar();   // every wave has written its slice of it
      const __amdgpu_buffer_rsrc_t ws_o_rsrc = __builtin_amdgcn_make_buffer_rsrc(p.ws_o, 0, p.ws_o_bytes, kBufferFormat);
      const __amdgpu_buffer_rsrc_t ws_lse_rsrc =
          __builtin_amdgcn_make_buffer_rsrc(p.ws_lse, 0, p.ws_lse_bytes, kBufferFormat);
      const float* po = reinterpret_cast<const float*>(piece_lds);
      const int rows = pub0.rows, row0 = 2 * pid * p.Rcap;
      for (int idx = ctid; idx < rows * (D / 4); idx += kCThreads) {
        const int r = idx / (D / 4);
        const int d4 = idx - r * (D / 4);
        const float l = po[rows * D + 2 * r + 1];
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(i32x4, *reinterpret_cast<const f32x4*>(po + r * D + 4 * d4) * (l > 0.f ? 1.f / l : 0.f)),
            ws_o_rsrc, ((row0 + r) * D + 4 * d4) * 4, 0, kDeviceCoherent);
      }
      for (int r = ctid; r < rows; r += kCThreads) {
        const float m = po[rows * D + 2 * r], l = po[rows * D + 2 * r + 1];
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, l > 0.f ? (m + log2f(l)) * kLn2 : -INFINITY),
                                              ws_lse_rsrc, (row0 + r) * 4, 0, kDeviceCoherent);
      }
      pub0.state = 0;
    }
    const bool due0 = pub0.state == 0 && v >= pub0.v + 2;
    const bool due1 = pub1.state == 0 && v >= pub1.v + 2;
    if (due0 || due1) {
      // Every consumer wave stored its own rows and d blocks of the piece:
      // each waits for its stores, then arrives on the piece's LDS counter,
      // and the last wave to arrive counts the piece on the unit's arrival
      // counter, after all eight waves' stores have completed.
      const int k = due0 ? 0 : 1;
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's piece stores
      int last = 0;
      if (lane == 0)
        last = __hip_atomic_fetch_add(&pub_arrive[k], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) ==
               kConsumers - 1;
      if (uniform(last)) {
        if (lane == 0)
          cnt[k] = __hip_atomic_fetch_add(p.counters + (k == 0 ? pub0 : pub1).unit, 1, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
        counted |= 1 << k;
      }
      (k == 0 ? pub0 : pub1).state = 1;
    }
    if (v >= count) continue;

    const int st = v & 1;
    gave_up |= !wait_count(&full_cnt[st], 2 * ((v >> 1) + 1), p.spin_limit);   // tile v is in stage st
    const int b = cur.b, kvh = cur.kvh, j = cur.j;
    const uint32_t s = cur.s;
    const int n = seq_tiles<C>(s);
    const int gt = g0 + v;
    const bool seg_first = v == 0 || j == 0;
    const bool seg_last = v == count - 1 || j == n - 1;
    if (seg_first) {
      roles(cur);
      m_run = -INFINITY;
      l_lane = 0.f;
      seg_g = gt;
    }

    {
      const char* ks = smem + st * C::kStage;
      const char* vs = ks + C::kLdsK;
      const int T = seq_T(s);
      const int hi = T - (n - 1 - j) * C::kTileKeys;
      const int lo = hi > C::kTileKeys ? hi - C::kTileKeys : 0;
      const int nk = hi - lo;
      const int lim = min(hi - 1, vis);   // this lane's row sees the keys <= lim of the tile
      // Key blocks kb0 and kb1 = kb0 + nks of the tile form a pair: two
      // independent score chains, one softmax step over their 8 keys per
      // lane, and (bf16) one 32-key P V contraction per d block.  A block
      // past the tile's keys reads staged rows that hold finite data and
      // is masked like any key >= hi.
      // (an inactive wave runs no pair)
      for (int kb0 = active ? kslot : C::kNKB; kb0 < C::kNKB; kb0 += 2 * nks) {
        if (kb0 * kBlk >= nk) break;
        const int key0 = lo + kb0 * kBlk;
        const int key1 = key0 + nks * kBlk;
        const int bstride = nks * kBlk * C::kPitchK;    // LDS bytes from block kb0 to kb1 (K)
        const int vbstride = nks * kBlk * C::kPitchV;   // (V)
        // S^T = K Q^T for 16 keys x 16 rows per block; lane (row lm,
        // quarter lg) gets the keys key + 4 lg + r, r = 0..3
        const char* krow = ks + (kb0 * kBlk + lm) * C::kPitchK + 16 * lg;
        // S^T chunk J of block h: kop(J, h) times Q chunk J
        auto score = [&](f32x4 acc, const u32x4& kop, int J) {
          if constexpr (W16) {
            return mfma32<ELT>(kop, qr[J], acc);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kop[e]), __uint_as_float(qr[J][e]), acc, 0,
                                                         0, 0);
            return acc;
          }
        };
        f32x4 sa[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
        if constexpr (C::kQJ <= 4) {
          // every K operand of the pair is read before the first score MFMA,
          // in the order the MFMAs take them, so the reads' latency is paid
          // once and each MFMA waits only for its own operand; the two
          // chains alternate
          u32x4 kop[C::kQJ][2];
#pragma unroll
          for (int J = 0; J < C::kQJ; ++J)
#pragma unroll
            for (int h = 0; h < 2; ++h) kop[J][h] = *reinterpret_cast<const u32x4*>(krow + h * bstride + 64 * J);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int J = 0; J < C::kQJ; ++J)
#pragma unroll
            for (int h = 0; h < 2; ++h) sa[h] = score(sa[h], kop[J][h], J);
        } else {
          // (f32, D = 128: twice the operand registers) one chain at a time
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            u32x4 kop[C::kQJ];
#pragma unroll
            for (int J = 0; J < C::kQJ; ++J) kop[J] = *reinterpret_cast<const u32x4*>(krow + h * bstride + 64 * J);
#pragma unroll
            for (int J = 0; J < C::kQJ; ++J) sa[h] = score(sa[h], kop[J], J);
          }
        }

        __builtin_amdgcn_sched_barrier(0);

        // V^T operands, read once the score MFMAs have taken their K
        // operands (fewer live registers; the reads overlap the MFMAs and the
        // softmax step): lane
        // (lm, lg) needs V rows key + 4 lg + e, e = 0..3, at d = 16 db + lm
        // of both blocks.  bf16: one transposed LDS read per block and d
        // block, in which lane t of the 16-lane group lg points at row
        // key + 4 lg + t / 4, columns 16 db + 4 (t % 4) .. + 3.
        i16x4 vt[W16 ? 2 * C::kDB : 1];
        if constexpr (W16) {
          typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
          const char* vrow = vs + (kb0 * kBlk + 4 * lg + (lm >> 2)) * C::kPitchV + 8 * (lm & 3);
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int db = 0; db < C::kDB; ++db)
              vt[h * C::kDB + db] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                  (lds_i16x4*)(__attribute__((address_space(3))) char*)(vrow + h * vbstride + 32 * db));
        }

        // mask, online softmax over the pair's keys (x: unscaled scores)
        float x[8];
        float mx = -INFINITY;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          // key kbase + 4 lg + r is masked when r > t (past the tile's keys
          // or past the row's last visible key); never inside the context
          const int t = lim - (h == 0 ? key0 : key1) - 4 * lg;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float xv = r > t ? -INFINITY : sa[h][r];
            x[4 * h + r] = xv;
            mx = fmaxf(mx, xv);
          }
        }
        if constexpr (TREE) {
          // a pair that reaches the draft region (the same for the whole
          // wave): key l_ctx + k is hidden unless bit k of the row's word is
          // set.  Keys past the tile's end are already hidden, and a key
          // that passed the compare has k < c_b <= 64.
          if (key1 + kBlk > l_ctx) {
            mx = -INFINITY;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int k = (h == 0 ? key0 : key1) + 4 * lg + r - l_ctx;
                if (k >= 0 && !((tmask >> (k & 63)) & 1u)) x[4 * h + r] = -INFINITY;
                mx = fmaxf(mx, x[4 * h + r]);
              }
            }
          }
        }
        mx = row_max(mx) * p.sl2;   // the scale is positive: max of the scaled scores
        // raise the running max only when the pair's max passes it by
        // more than kLazyMax; the four lanes of a row decide alike
        const bool raise = mx > m_run + kLazyMax;
        if (__any(raise)) {
          const float m_new = raise ? mx : m_run;
          const float alpha = __builtin_amdgcn_exp2f(m_run - (m_new == -INFINITY ? 0.f : m_new));
          l_lane *= alpha;
#pragma unroll
          for (int db = 0; db < C::kDB; ++db) o[db] *= alpha;
          m_run = m_new;
        }
        const float m_use = m_run == -INFINITY ? 0.f : m_run;
        float pr[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          pr[r] = __builtin_amdgcn_exp2f(fmaf(x[r], p.sl2, -m_use));
          l_lane += pr[r];
        }

        // O^T += V^T P^T
        if constexpr (W16) {
          // 32-key contraction: element e of a lane's operands is key
          // 4 lg + e of block kb0 (e < 4) or key 4 lg + e - 4 of kb1
          const u32x4 pb = pack_p<ELT>(pr);
#pragma unroll
          for (int db = 0; db < C::kDB; ++db) {
            const i16x4 a0 = vt[db], a1 = vt[C::kDB + db];
            const u32x4 va = {__builtin_bit_cast(uint2, a0).x, __builtin_bit_cast(uint2, a0).y,
                              __builtin_bit_cast(uint2, a1).x, __builtin_bit_cast(uint2, a1).y};
            o[db] = mfma32<ELT>(va, pb, o[db]);
          }
        } else {
          // f32: lane (lm, lg) takes V rows key + 4 lg + r at d = 16 db + lm
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const char* vrow = vs + (kb0 * kBlk + 4 * lg) * C::kPitchV + h * vbstride + 4 * lm;
#pragma unroll
            for (int db = 0; db < C::kDB; ++db)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                o[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                    *reinterpret_cast<const float*>(vrow + r * C::kPitchV + 64 * db), pr[4 * h + r], o[db], 0, 0, 0);
          }
        }
      }
    }

    if (!seg_last) {
      signal_count(&empty_cnt[st]);   // done with stage st
    } else {
      // the next segment's Q (loaded a segment ago) becomes current before
      // this segment's results are stored, so its wait covers no store
#pragma unroll
      for (int J = 0; J < C::kQJ; ++J) qr[J] = qn[J];
#pragma unroll
      for (int J = 0; J < C::kQJ; ++J) asm volatile("" : "+v"(qr[J])::"memory");
      if constexpr (TREE) {
        tm_r = tm_n;
        asm volatile("" : "+v"(tm_r)::"memory");
      }
      // the Q of the segment after next is loaded now, right after qn was
      // read, and before this segment's stores
      {
        int v1;
        const Cursor c1 = next_segment(cur, v, v1);
        if (v1 < count) {
          int v2;
          const Cursor c2 = next_segment(c1, v1, v2);
          if (v2 < count) load_q(c2, qn, tm_n);
        }
      }
      // ---- combine the key-split states of each row block in one LDS
      // round: every wave of the row block writes its (max, sum, O) state,
      // then each merges all of them for its own slice of d blocks.  This
      // tile's stage is the scratch; it is released only afterwards.
      float fm = m_run, fl = row_sum(l_lane);   // this lane's row: max (log2 units) and sum
      const int s_db = nks <= C::kDB ? C::kDB / nks : 1;
      const int d_lo = kslot * s_db, d_hi = d_lo + s_db;   // this wave's d blocks
      const int unit_first = gt - j;                 // global index of the unit's tile 0
      const bool whole = seg_g == unit_first && j == n - 1;
      // The piece of the range's first segment is held in LDS and stored
      // only at the range's last tile, when it fits there and more tiles
      // follow: stores issued while the range's tiles stream in slow the rest
      // of the stream down, stores late in it much less.  It is written by
      // the key-split merge below (units of one or two row blocks), not yet
      // normalised: O rows, then (max, sum) per row.  (Those units' waves
      // pass consumer barriers at each unit end, so by then the cost sums
      // that share the LDS are no longer read.)
      const bool hold =
          HOLD && !whole && seg_g == g0 && v + 1 < count && nks > 1 && R * (D + 2) * 4 <= C::kPieceLds;
      if (nks > 1) {
        char* merge_lds = smem + st * C::kStage;
        cbar();   // every consumer is done with this tile's stage
        if (active) {
          const int region = rb * nks + kslot;
          f32x4* reg = reinterpret_cast<f32x4*>(merge_lds + region * (64 * D));
          // the d blocks the other waves of the row block merge (this wave
          // keeps its own slice in registers)
#pragma unroll
          for (int db = 0; db < C::kDB; ++db)
            if (db < d_lo || db >= d_hi) reg[db * 64 + lane] = o[db];
          if (lg == 0) {   // the four lanes of a row hold the same values
            mst[region][0][lm] = m_run;
            mst[region][1][lm] = fl;
          }
        }
        cbar();
        if (active) {
          // the same order of operations in every wave of the row block
          float M = -INFINITY;
          for (int k = 0; k < nks; ++k) M = fmaxf(M, mst[rb * nks + k][0][lm]);
          const float Mu = M == -INFINITY ? 0.f : M;
          float wk[kConsumers];
          float L = 0.f;
#pragma unroll
          for (int k = 0; k < kConsumers; ++k) {
            if (k < nks) {
              wk[k] = __builtin_amdgcn_exp2f(mst[rb * nks + k][0][lm] - Mu);
              L += mst[rb * nks + k][1][lm] * wk[k];
            }
          }
          fm = M;
          fl = L;
#pragma unroll
          for (int db = 0; db < C::kDB; ++db) {
            if (db >= d_lo && db < d_hi) {
              f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
              for (int k = 0; k < kConsumers; ++k) {
                if (k < nks) {
                  const f32x4* reg = reinterpret_cast<const f32x4*>(merge_lds + (rb * nks + k) * (64 * D));
                  acc += (k == kslot ? o[db] : reg[db * 64 + lane]) * wk[k];
                }
              }
              o[db] = acc;
              if (hold && row_valid)
                *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(piece_lds) + row * D + 16 * db + 4 * lg) = acc;
            }
          }
          if (hold && row_valid && kslot == 0 && lg == 0) {
            float* ps = reinterpret_cast<float*>(piece_lds) + R * D + 2 * row;
            ps[0] = M;
            ps[1] = L;
          }
        }
      }
      signal_count(&empty_cnt[st]);   // done with stage st (and its scratch use)

      // ---- this wave's slice of the result, stored at the top of the next
      // iteration: the whole unit (final result) or a piece of it
      pend = true;
      pend_whole = whole;
      pend_ok = active && row_valid;
      pend_inv = fl > 0.f ? 1.f / fl : 0.f;
      pend_lse = fl > 0.f ? (fm + log2f(fl)) * kLn2 : -INFINITY;
      pend_row = whole ? (b * p.C_max + tok) * p.Hq + kvh * g + row - tok * g
                       : (2 * pid + (seg_g == g0 ? 0 : 1)) * p.Rcap + row;
      if (!whole) {
        Pub q;
        q.state = 0;
        q.unit = b * Hkv + kvh;
        q.v = v + 1;   // the iteration that stores it
        q.rows = R;
        // The piece of the range's first segment is held in LDS and stored
        // only at the range's last tile, when it fits there and more tiles
        // follow: stores issued while the range's tiles stream in slow the
        // rest of the stream down (measured), stores late in it much less.
        // (Units with one or two row blocks: their waves pass consumer
        // barriers at each unit end, so the cost sums are no longer read.)
        if (hold) {
          pend_ok = false;   // written to LDS by the key-split merge above
          q.state = 3;
          // the iteration that stores it: three quarters into the range, so
          // that it has arrived when the previous range, which merges the
          // unit, ends (a store that early costs the stream less than that
          // merge's wait; halfway and seven eighths in measured slower)
          q.v = min(count - 1, max(v + 1, (3 * count) / 4));
        }
        {
          if (v == count - 1 && unit_first >= g0) {
            pend_direct = true;
            pend_k = n_pub;
            q.state = 2;   // not published in the loop
            if (wc == 0 && lane == 0)
              probe = __hip_atomic_load(p.counters + q.unit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
        }
        if (n_pub == 0) pub0 = q;
        else pub1 = q;
        ++n_pub;
      }
    }
    if (v + 1 < count) advance(cur);
  }

  // ---- the last segment's piece kept in registers: merged with the next
  // range's piece (its first segment, slot 2 (pid + 1)) into the final rows
  // when that was the unit's only other piece and it had arrived at the last
  // tile, else stored and counted.  (Merging there saves the piece's store,
  // its count and a read back at the end of the launch, when nothing else
  // hides them: the next range publishes its piece early.)
  {
    if (pend_direct) {
      // two pieces, the other one arrived (wave 0 wrote sh_share itself;
      // the other waves read it after the barrier)
      if (wc == 0 && lane == 0) sh_direct = sh_share[1][2] == pid + 1 && probe == 1 ? 1 : 0;
      cbar();
      const int u = sh_share[1][0], ql = sh_share[1][2];
      const __amdgpu_buffer_rsrc_t ws_o_rsrc =
          __builtin_amdgcn_make_buffer_rsrc(p.ws_o, 0, p.ws_o_bytes, kBufferFormat);
      const __amdgpu_buffer_rsrc_t ws_lse_rsrc =
          __builtin_amdgcn_make_buffer_rsrc(p.ws_lse, 0, p.ws_lse_bytes, kBufferFormat);
      const int s_db = nks <= C::kDB ? C::kDB / nks : 1;
      const int d_lo = kslot * s_db, d_hi = d_lo + s_db;   // this wave's d blocks
      if (sh_direct) {
        if (pend_ok) {
          const int srow = 2 * ql * p.Rcap + row;
          const float lp = __builtin_bit_cast(
              float, __builtin_amdgcn_raw_buffer_load_b32(ws_lse_rsrc, srow * 4, 0, kDeviceCoherent));
          f32x4 xp[C::kDB];
#pragma unroll
          for (int db = 0; db < C::kDB; ++db)
            if (db >= d_lo && db < d_hi)
              xp[db] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                     ws_o_rsrc, (srow * D + 16 * db + 4 * lg) * 4, 0, kDeviceCoherent));
          // this range's piece, then the next range's, as the merge of
          // pieces takes them
          float m = -INFINITY, z = 0.f, wa = 0.f, wb = 0.f;
          if (pend_lse != -INFINITY) {
            m = pend_lse;
            z = 1.f;
            wa = 1.f;
          }
          if (lp != -INFINITY) {
            const float nm = fmaxf(m, lp);
            const float a = expf(m - nm);
            const float w = expf(lp - nm);
            z = z * a + w;
            wa *= a;
            wb = w;
            m = nm;
          }
          const float inv_z = z > 0.f ? 1.f / z : 0.f;
          // (cur is still the last tile's cursor)
          const int pend_orow = (cur.b * p.C_max + tok) * p.Hq + cur.kvh * g + row - tok * g;
          float* dst = p.out + (size_t)pend_orow * D;
#pragma unroll
          for (int db = 0; db < C::kDB; ++db)
            if (db >= d_lo && db < d_hi)
            {
              const f32x4 res = (o[db] * pend_inv * wa + wb * xp[db]) * inv_z;
              if constexpr (NT) __builtin_nontemporal_store(res, reinterpret_cast<f32x4*>(dst + 16 * db + 4 * lg));
              else *reinterpret_cast<f32x4*>(dst + 16 * db + 4 * lg) = res;
            }
          if (kslot == 0 && lg == 0) {
            const float res_lse = z > 0.f ? m + logf(z) : -INFINITY;
            if constexpr (NT) __builtin_nontemporal_store(res_lse, p.lse + pend_orow);
            else p.lse[pend_orow] = res_lse;
          }
        }
        if (ctid == 0) __hip_atomic_store(p.counters + u, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      } else {
        if (pend_ok) {
          if (kslot == 0 && lg == 0)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, pend_lse), ws_lse_rsrc, pend_row * 4, 0,
                                                  kDeviceCoherent);
#pragma unroll
          for (int db = 0; db < C::kDB; ++db)
            if (db >= d_lo && db < d_hi)
              __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, o[db] * pend_inv), ws_o_rsrc,
                                                     (pend_row * D + 16 * db + 4 * lg) * 4, 0, kDeviceCoherent);
        }
        // counted as in the loop: after every wave's stores, by the last wave
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        int last = 0;
        if (lane == 0)
          last = __hip_atomic_fetch_add(&pub_arrive[pend_k], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) ==
                 kConsumers - 1;
        if (uniform(last)) {
          if (lane == 0) {
            const int c = __hip_atomic_fetch_add(p.counters + u, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (pend_k == 0) cnt[0] = c;   // (constant indices keep cnt in registers)
            else cnt[1] = c;
          }
          counted |= 1 << pend_k;
        }
      }
    }
  }

  // ---- merges of cut units, now that this workgroup's tiles are done.  The
  // wave that counted piece k sets its flag (sh_flag starts at 0: no merge
  // here; else 1 + the entry of sh_share for the unit); that wave arrived
  // last on the piece's LDS counter, after wave 0 had written sh_share.
  // (Units merged from registers above are not counted here.)  With HOLD
  // the last piece to arrive merges its unit.  Otherwise the unit is merged
  // by the first of its holders to finish its own tiles once all pieces have
  // arrived: it claims the unit by switching the counter from np to np |
  // kClaimed, a compare-and-swap that fails while pieces are missing (a
  // later holder then succeeds), once the unit is claimed, and after its
  // merge has reset the counter to 0.  (The last piece to arrive was often
  // the last range to finish, whose merges then ended the launch.)
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    if ((counted >> k) & 1) {
      const Pub& q = k == 0 ? pub0 : pub1;
      const int e = q.unit == sh_share[0][0] ? 0 : 1;
      const int np = sh_share[e][2] - sh_share[e][1] + 1;   // pieces of the unit
      if (lane == 0) {
        bool mine;
        if constexpr (HOLD) {
          mine = cnt[k] + 1 == np;
        } else {
          int expected = np;
          mine = __hip_atomic_compare_exchange_strong(p.counters + q.unit, &expected, np | kClaimed, __ATOMIC_RELAXED,
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        sh_flag[k] = mine ? 1 + e : 0;
      }
    }
  }
  cbar();
  {
    const int f0 = sh_flag[0], f1 = sh_flag[1];
    if (f0 || f1)
      merge_units<D, NT>(p, seqs, ctid, sh_share[f0 ? f0 - 1 : 0], sh_share[f1 ? f1 - 1 : 0], f0 != 0, f1 != 0);
  }
  report_give_up(gave_up);
}

// Zero the per-unit counters of a workspace.
__global__ void zero_counters_kernel(int* counters, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) counters[i] = 0;
}

// ---------------------------------------------------------------- host side

int elt_bytes(int dtype) { return dtype == SPECMOE_F32 ? 4 : 2; }

bool known_dtype(int dtype) { return dtype == SPECMOE_F32 || dtype == SPECMOE_BF16 || dtype == SPECMOE_F16; }

int key_tile(int dtype, int D) {
  const int elt = elt_bytes(dtype);
  return kHalf / (D * elt);
}

// Workspace layout: a 256-byte header holding the sticky status word, the
// per-unit arrival counters for the largest launch (same offsets for every
// descriptor with the same Hkv), then the partial results of the pieces, two
// slots per workgroup.  The header and the counters form the zeroed region.
constexpr size_t kHeaderBytes = 256;
struct Plan {
  int g, P, Rcap;
  size_t zero_bytes;   // header + counters
  size_t slots, ws_lse_off, ws_o_off, ws_bytes;
};

int validate_desc(const specmoe_verify_desc* d) {
  if (!d) return SPECMOE_ERR_NULL_POINTER;
  if (!known_dtype(d->dtype)) return SPECMOE_ERR_DTYPE;
  if (d->D != 64 && d->D != 128) return SPECMOE_ERR_HEAD_DIM;
  if (d->B < 0 || d->Hq <= 0 || d->Hkv <= 0 || d->C_max < 1 || d->S_max < d->C_max)
    return SPECMOE_ERR_SHAPE;
  if (d->Hq % d->Hkv != 0) return SPECMOE_ERR_GQA;
  const int64_t g = d->Hq / d->Hkv;
  if ((int64_t)d->C_max * g > kMaxRows) return SPECMOE_ERR_ROWS;
  if ((d->flags & ~SPECMOE_FLAG_NO_WAIT) != 0) return SPECMOE_ERR_FLAGS;
  if (d->grid_blocks < 0 || d->grid_blocks > kMaxGrid) return SPECMOE_ERR_GRID;
  // partial results are addressed through 32-bit buffer descriptors
  const int64_t grid = d->grid_blocks ? d->grid_blocks : kDefaultGrid;
  if (2 * grid * (int64_t)d->C_max * g * d->D * 4 >= ((int64_t)1 << 31)) return SPECMOE_ERR_GRID;
  // index arithmetic: (sequence, token, head) row indices stay in 32 bits,
  // byte offsets inside one (sequence, KV head) slab are 32-bit, packed
  // sequence lengths need T < 2^24, tile counts per launch stay in 32 bits.
  if ((int64_t)d->B * d->C_max * d->Hq >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  const int64_t elt = elt_bytes(d->dtype);
  if ((int64_t)d->S_max * d->D * elt >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  if (d->S_max >= (1 << 24)) return SPECMOE_ERR_SHAPE;
  const int64_t tile = key_tile(d->dtype, d->D);
  if ((int64_t)kMaxSeqs * d->Hkv * ((d->S_max + tile - 1) / tile) >= ((int64_t)1 << 30)) return SPECMOE_ERR_SHAPE;
  // the per-KV-head tile cost prefix of the schedule fits in 32 bits
  const int64_t w_hi = kTileCost + (d->C_max * g + kBlk - 1) / kBlk + kExtraMax;
  if ((int64_t)kMaxSeqs * ((d->S_max + tile - 1) / tile) * w_hi >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  return SPECMOE_OK;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

Plan make_plan(const specmoe_verify_desc* d) {
  Plan pl;
  pl.g = d->Hq / d->Hkv;
  pl.P = d->grid_blocks ? d->grid_blocks : kDefaultGrid;
  pl.Rcap = d->C_max * pl.g;
  pl.zero_bytes = kHeaderBytes + align256((size_t)kMaxSeqs * d->Hkv * sizeof(int));
  pl.slots = (size_t)2 * pl.P;
  pl.ws_lse_off = pl.zero_bytes;
  pl.ws_o_off = pl.ws_lse_off + align256(pl.slots * pl.Rcap * sizeof(float));
  pl.ws_bytes = pl.ws_o_off + pl.slots * pl.Rcap * d->D * sizeof(float);
  return pl;
}

// Results (out and lse) are stored write-back, except in launches with both
// many units per workgroup (at least kNtUnitsPerWg) and a large output (at
// least kNtOutBytes), where the workgroups store results many times while the
// K/V stream runs: there the non-temporal policy measured faster (B = 256, 8
// KV heads, 16-33 MB of output: 2-7%; B = 128, 10.5 MB: 1.4%), while launches
// with fewer, larger units (ragged chunks, tree drafts, B = 64) or a small
// output (one-token decode) were 1-5% slower with it.  Launches that hold
// their first piece in LDS keep that variant.
constexpr int kNtUnitsPerWg = 4;
constexpr size_t kNtOutBytes = (size_t)8 << 20;

template <int ELT, int D, bool TREE, bool PAGED>
void launch(Params p, const Plan& pl, hipStream_t stream) {
  using C = Cfg<ELT != kF32, D>;
  // units of at most two 16-row blocks whose piece fits the LDS left beside
  // the stages hold their range's first piece there
  const bool hold = p.Rcap <= 2 * kBlk && p.Rcap * (D + 2) * 4 <= C::kPieceLds;
  const int B = p.B;
  // batches beyond kMaxSeqs sequences run as consecutive launches on the stream
  for (int b0 = 0; b0 < B; b0 += kMaxSeqs) {
    Params s = p;
    s.B = B - b0 < kMaxSeqs ? B - b0 : kMaxSeqs;
    s.q = p.q + (size_t)b0 * p.C_max * p.Hq * C::kRowBytes;
    if (PAGED) {
      s.block_table = p.block_table + (size_t)b0 * p.pages_per_seq;
    } else {
      const size_t slab = (size_t)b0 * p.Hkv * p.S_max * C::kRowBytes;
      s.k = p.k + slab;
      s.v = p.v + slab;
    }
    s.ctx_lens = p.ctx_lens + b0;
    s.chunk_lens = p.chunk_lens + b0;
    if (TREE) s.draft_mask = p.draft_mask + (size_t)b0 * p.C_max;
    s.out = p.out + (size_t)b0 * p.C_max * p.Hq * D;
    s.lse = p.lse + (size_t)b0 * p.C_max * p.Hq;
    const bool nt = s.B * p.Hkv >= kNtUnitsPerWg * pl.P &&
                    (size_t)s.B * p.C_max * p.Hq * (D + 1) * sizeof(float) >= kNtOutBytes;
    if (hold)
      hipLaunchKernelGGL((verify_attn_kernel<ELT, D, TREE, PAGED, kModeHold>), dim3(pl.P), dim3(kThreads), 0, stream, s);
    else if (nt)
      hipLaunchKernelGGL((verify_attn_kernel<ELT, D, TREE, PAGED, kModeNt>), dim3(pl.P), dim3(kThreads), 0, stream, s);
    else
      hipLaunchKernelGGL((verify_attn_kernel<ELT, D, TREE, PAGED, kModePlain>), dim3(pl.P), dim3(kThreads), 0, stream, s);
  }
}

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

template <int ELT, bool PAGED>
void launch_for_elt(int D, bool tree, const Params& p, const Plan& pl, hipStream_t s) {
  if (tree) {
    if (D == 128) launch<ELT, 128, true, PAGED>(p, pl, s);
    else launch<ELT, 64, true, PAGED>(p, pl, s);
  } else {
    if (D == 128) launch<ELT, 128, false, PAGED>(p, pl, s);
    else launch<ELT, 64, false, PAGED>(p, pl, s);
  }
}

template <bool PAGED>
void launch_for_paging(int dtype, int D, bool tree, const Params& p, const Plan& pl, hipStream_t s) {
  if (dtype == SPECMOE_BF16) launch_for_elt<kBF16, PAGED>(D, tree, p, pl, s);
  else if (dtype == SPECMOE_F16) launch_for_elt<kF16, PAGED>(D, tree, p, pl, s);
  else launch_for_elt<kF32, PAGED>(D, tree, p, pl, s);
}

void launch_for(int dtype, int D, bool tree, bool paged, const Params& p, const Plan& pl, hipStream_t s) {
  if (paged) launch_for_paging<true>(dtype, D, tree, p, pl, s);
  else launch_for_paging<false>(dtype, D, tree, p, pl, s);
}

// Host checks and launch of both entry points; draft_mask is NULL for a
// chain draft.
// Page geometry of a paged call: page_size a power of two in [8, 65536]
// (tiles hold at most 256 keys, so a tile meets at most 33 pages, one per
// producer lane), S_max = page_size * pages_per_seq, a non-empty pool.
int validate_pages(const specmoe_verify_desc* d, const specmoe_paged_kv* pk) {
  if (!pk) return SPECMOE_ERR_NULL_POINTER;
  const int ps = pk->page_size;
  if (ps < 8 || ps > 65536 || (ps & (ps - 1)) != 0) return SPECMOE_ERR_PAGES;
  if (pk->pages_per_seq < 1 || pk->num_pages < 1) return SPECMOE_ERR_PAGES;
  if ((int64_t)ps * pk->pages_per_seq != d->S_max) return SPECMOE_ERR_PAGES;
  if ((int64_t)kMaxSeqs * pk->pages_per_seq >= ((int64_t)1 << 31)) return SPECMOE_ERR_PAGES;
  return SPECMOE_OK;
}

int run(const void* q, const void* k_cache, const void* v_cache, const int32_t* ctx_lens,
        const int32_t* chunk_lens, const uint64_t* draft_mask, bool tree, float scale, float* out, float* lse,
        void* stream, const specmoe_verify_desc* desc, const int32_t* block_table = nullptr,
        const specmoe_paged_kv* paged = nullptr, bool clear_counters = false) {
  const int st = validate_desc(desc);
  if (st != SPECMOE_OK) return st;
  if (tree && desc->C_max > kMaxDraftBits) return SPECMOE_ERR_MASK;
  const bool is_paged = paged != nullptr;
  if (is_paged) {
    const int sp = validate_pages(desc, paged);
    if (sp != SPECMOE_OK) return sp;
  }
  if (desc->B == 0) return SPECMOE_OK;   // nothing to read or write
  if (!q || !k_cache || !v_cache || !ctx_lens || !chunk_lens || !out || !lse) return SPECMOE_ERR_NULL_POINTER;
  if (tree && !draft_mask) return SPECMOE_ERR_NULL_POINTER;
  if (!(scale > 0.f) || !isfinite(scale)) return SPECMOE_ERR_SCALE;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out)) return SPECMOE_ERR_ALIGN;
  if (tree && (reinterpret_cast<uintptr_t>(draft_mask) & 7u) != 0) return SPECMOE_ERR_ALIGN;
  if (is_paged && !block_table) return SPECMOE_ERR_NULL_POINTER;
  const Plan pl = make_plan(desc);
  if (!desc->workspace) return SPECMOE_ERR_NULL_POINTER;
  if (!aligned16(desc->workspace)) return SPECMOE_ERR_ALIGN;
  if (desc->workspace_bytes < pl.ws_bytes) return SPECMOE_ERR_WORKSPACE;

  Params p;
  p.q = static_cast<const char*>(q);
  p.k = static_cast<const char*>(k_cache);
  p.v = static_cast<const char*>(v_cache);
  p.ctx_lens = ctx_lens;
  p.chunk_lens = chunk_lens;
  p.out = out;
  p.lse = lse;
  p.draft_mask = draft_mask;
  p.block_table = block_table;
  p.page_shift = is_paged ? __builtin_ctz((unsigned)paged->page_size) : 0;
  p.pages_per_seq = is_paged ? paged->pages_per_seq : 0;
  p.num_pages = is_paged ? paged->num_pages : 0;
  char* ws = static_cast<char*>(desc->workspace);
  p.status = reinterpret_cast<int*>(ws);
  p.spin_limit = (desc->flags & SPECMOE_FLAG_NO_WAIT) ? 0 : kSpinLimit;
  p.counters = reinterpret_cast<int*>(ws + kHeaderBytes);
  p.ws_lse = reinterpret_cast<float*>(ws + pl.ws_lse_off);
  p.ws_o = reinterpret_cast<float*>(ws + pl.ws_o_off);
  p.ws_lse_bytes = (int)(pl.ws_o_off - pl.ws_lse_off);
  p.ws_o_bytes = (int)(pl.ws_bytes - pl.ws_o_off);
  p.B = desc->B;
  p.Hq = desc->Hq;
  p.Hkv = desc->Hkv;
  p.g = pl.g;
  p.C_max = desc->C_max;
  p.S_max = desc->S_max;
  p.Rcap = pl.Rcap;
  p.P = pl.P;
  p.sl2 = scale * kLog2e;

  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();  // clear a stale error from unrelated work
  if (clear_counters) {
    // the arrival counters of the units of one launch (at most kMaxSeqs
    // sequences), zeroed by a small kernel ahead of the main one
    const int n = (desc->B < kMaxSeqs ? desc->B : kMaxSeqs) * desc->Hkv;
    hipLaunchKernelGGL(zero_counters_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p.counters, n);
  }
  launch_for(desc->dtype, desc->D, tree, is_paged, p, pl, s);
  if (hipGetLastError() != hipSuccess) return SPECMOE_ERR_LAUNCH;
  return SPECMOE_OK;
}

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_for_current_device(void** ptr_out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SPECMOE_ERR_LAUNCH;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return SPECMOE_ERR_LAUNCH;
    g_scratch_ptr[dev] = ptr;
  }
  *ptr_out = g_scratch_ptr[dev];
  return SPECMOE_OK;
}

}  // namespace

extern "C" {

size_t specmoe_verify_attn_workspace_bytes(const specmoe_verify_desc* desc) {
  if (validate_desc(desc) != SPECMOE_OK) return 0;
  return make_plan(desc).ws_bytes;
}

int specmoe_verify_attn_workspace_init(void* workspace, size_t workspace_bytes, void* stream,
                                       const specmoe_verify_desc* desc) {
  const int st = validate_desc(desc);
  if (st != SPECMOE_OK) return st;
  if (!workspace) return SPECMOE_ERR_NULL_POINTER;
  if (!aligned16(workspace)) return SPECMOE_ERR_ALIGN;
  const Plan pl = make_plan(desc);
  if (workspace_bytes < pl.ws_bytes) return SPECMOE_ERR_WORKSPACE;
  const int n = (int)(pl.zero_bytes / sizeof(int));
  (void)hipGetLastError();
  hipLaunchKernelGGL(zero_counters_kernel, dim3((n + 255) / 256), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<int*>(workspace), n);
  return hipGetLastError() == hipSuccess ? SPECMOE_OK : SPECMOE_ERR_LAUNCH;
}

int specmoe_verify_attn_status(const void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace && workspace_bytes == 0) {   // the current device's static scratch
    void* ptr = nullptr;
    const int st = scratch_for_current_device(&ptr);
    if (st != SPECMOE_OK) return st;
    workspace = ptr;
    workspace_bytes = kScratchBytes;
  }
  if (!workspace) return SPECMOE_ERR_NULL_POINTER;
  if (!aligned16(workspace)) return SPECMOE_ERR_ALIGN;
  if (workspace_bytes < kHeaderBytes) return SPECMOE_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int word = 0;
  (void)hipGetLastError();
  if (hipMemcpyAsync(&word, workspace, sizeof(word), hipMemcpyDeviceToHost, s) != hipSuccess)
    return SPECMOE_ERR_LAUNCH;
  if (hipStreamSynchronize(s) != hipSuccess) return SPECMOE_ERR_LAUNCH;
  return (word & kGaveUp) ? SPECMOE_ERR_HANDOFF : SPECMOE_OK;
}

int32_t specmoe_verify_attn_key_tile(const specmoe_verify_desc* desc) {
  if (!desc) return SPECMOE_ERR_NULL_POINTER;
  if (!known_dtype(desc->dtype)) return SPECMOE_ERR_DTYPE;
  if (desc->D != 64 && desc->D != 128) return SPECMOE_ERR_HEAD_DIM;
  return key_tile(desc->dtype, desc->D);
}

const char* specmoe_status_str(int status) {
  switch (status) {
    case SPECMOE_OK: return "ok";
    case SPECMOE_ERR_NULL_POINTER: return "null pointer argument";
    case SPECMOE_ERR_SHAPE: return "invalid shape (B, Hq, Hkv, C_max, S_max) or sizes too large";
    case SPECMOE_ERR_GQA: return "Hq is not a multiple of Hkv";
    case SPECMOE_ERR_HEAD_DIM: return "unsupported head dimension (must be 64 or 128)";
    case SPECMOE_ERR_DTYPE: return "unsupported dtype";
    case SPECMOE_ERR_ROWS: return "C_max * (Hq / Hkv) exceeds 128 query rows per KV head";
    case SPECMOE_ERR_GRID: return "grid_blocks must be 0 (default) or in [1, 2048], with partial results under 2 GB";
    case SPECMOE_ERR_FLAGS: return "flags may only hold SPECMOE_FLAG_NO_WAIT";
    case SPECMOE_ERR_WORKSPACE: return "workspace too small";
    case SPECMOE_ERR_ALIGN: return "q, k_cache, v_cache, out and workspace must be 16-byte aligned";
    case SPECMOE_ERR_SCALE: return "scale must be finite and positive";
    case SPECMOE_ERR_LAUNCH: return "HIP kernel launch failed";
    case SPECMOE_ERR_MASK: return "draft masks hold at most 64 draft tokens: C_max must be <= 64";
    case SPECMOE_ERR_HANDOFF: return "an in-kernel wait for another wave gave up: results of a call are unspecified";
    case SPECMOE_ERR_PAGES:
      return "page_size must be a power of two in [8, 65536], pages_per_seq and num_pages positive, "
             "S_max = page_size * pages_per_seq";
    default: return "unknown status";
  }
}

int specmoe_verify_attn(const void* q, const void* k_cache, const void* v_cache, const int32_t* ctx_lens,
                        const int32_t* chunk_lens, float scale, float* out, float* lse, void* stream,
                        const specmoe_verify_desc* desc) {
  return run(q, k_cache, v_cache, ctx_lens, chunk_lens, nullptr, false, scale, out, lse, stream, desc);
}

int specmoe_verify_attn_noalloc(const void* q, const void* k_cache, const void* v_cache, const int32_t* ctx_lens,
                                const int32_t* chunk_lens, float scale, float* out, float* lse, void* stream,
                                const specmoe_verify_desc* desc) {
  const int st = validate_desc(desc);
  if (st != SPECMOE_OK) return st;
  if (make_plan(desc).ws_bytes > kScratchBytes) return SPECMOE_ERR_WORKSPACE;
  if (desc->B == 0) return SPECMOE_OK;
  void* ws = nullptr;
  const int ss = scratch_for_current_device(&ws);
  if (ss != SPECMOE_OK) return ss;
  specmoe_verify_desc d = *desc;
  d.workspace = ws;
  d.workspace_bytes = kScratchBytes;
  return run(q, k_cache, v_cache, ctx_lens, chunk_lens, nullptr, false, scale, out, lse, stream, &d, nullptr, nullptr,
             true);
}

int specmoe_verify_attn_tree(const void* q, const void* k_cache, const void* v_cache, const int32_t* ctx_lens,
                             const int32_t* chunk_lens, const uint64_t* draft_mask, float scale, float* out,
                             float* lse, void* stream, const specmoe_verify_desc* desc) {
  return run(q, k_cache, v_cache, ctx_lens, chunk_lens, draft_mask, true, scale, out, lse, stream, desc);
}

int specmoe_verify_attn_paged(const void* q, const void* k_pages, const void* v_pages, const int32_t* block_table,
                              const int32_t* ctx_lens, const int32_t* chunk_lens, const uint64_t* draft_mask,
                              float scale, float* out, float* lse, void* stream, const specmoe_verify_desc* desc,
                              const specmoe_paged_kv* paged) {
  if (!paged) return SPECMOE_ERR_NULL_POINTER;
  return run(q, k_pages, v_pages, ctx_lens, chunk_lens, draft_mask, draft_mask != nullptr, scale, out, lse, stream,
             desc, block_table, paged);
}

}  // extern "C"
