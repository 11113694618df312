// Chunked verification attention for MI355X (gfx950, CDNA4).
//
// Computes, for every sequence b and KV head, softmax(scale*Q K^T + M) V over
// the cached context plus the draft chunk, with a chain mask inside the chunk
// (SpecMoEOff, Section 5.1), and the log-sum-exp of every row.
//
// Design (one kernel launch per call):
//   * Unit of work = (sequence b, KV head).  The c_b draft tokens times the g
//     query heads that share the KV head form the unit's R_b = c_b*g query
//     rows; they are packed into 32-row MFMA tiles, so Q K^T and P V become
//     small dense contractions that reuse every K/V byte for all rows.
//   * Key tiles: a unit's keys [0, T_b) are cut into tiles of kTileKeys keys
//     anchored at T_b (tile n-1 = [T_b - kTileKeys, T_b)), so the chunk's own
//     keys always sit in the unit's last tile and every tile holds a key that
//     every query row of the unit can see.
//   * Stream-K schedule: the tiles of all units, in unit order, form one list
//     that is cut into equal contiguous ranges, one per persistent workgroup
//     (2 per CU).  Every workgroup streams the same number of K/V bytes, so no
//     CU idles at the end of the launch.  A unit cut by a range boundary is a
//     sequence-wise KV partition whose partial results must be combined, as
//     the paper notes for its sequence-dimension KV split (Section 5.2): each
//     piece writes (O/l, lse) to the workspace, counts itself on an atomic
//     arrival counter, and the last piece to arrive merges all of them with
//     log-sum-exp weights.  Uncut units write their result directly.
//   * K/V streaming: each iteration stages a 32 KB K tile and a 32 KB V tile
//     in LDS with fully coalesced 16-byte loads (one wave instruction reads
//     1 KB of contiguous cache rows); the next tile's loads are in flight in
//     registers while the current tile is consumed.  LDS rows are padded by
//     16 bytes, so every MFMA operand read is free of bank conflicts and all
//     operand addresses are a per-lane base plus an immediate.
//   * Scores are formed transposed, S^T = K Q^T (keys on the MFMA M side,
//     query rows on N), so each lane holds one query row: the online-softmax
//     row statistics are per-lane scalars, row reductions need one cross-lane
//     step (lanes l and l^32), and the probabilities are already in the B
//     operand layout of O^T = V^T P^T.
//   * bf16 inputs use v_mfma_f32_32x32x16_bf16 with fp32 accumulation (P is
//     rounded to bf16 for the PV product); f32 inputs use v_mfma_f32_32x32x2_f32.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "specmoe_verify.h"

namespace {

constexpr int kThreads = 256;        // 4 waves of 64
constexpr int kWaves = 4;
constexpr int kSub = 32;             // keys per MFMA subtile
constexpr int kRowTile = 32;         // query rows per MFMA tile
constexpr int kMaxRows = 128;        // row tiles per unit <= 4
constexpr int kTileBytes = 32768;    // K bytes (and V bytes) staged per iteration
constexpr int kDefaultGrid = 512;    // persistent workgroups: 2 per CU on MI355X's 256 CUs
constexpr int kMaxSeqs = 2048;       // sequences per launch (their lengths live in LDS)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) short i16x8;
typedef __attribute__((ext_vector_type(4))) int i32x4;

// Cache policy of the partial-result buffer accesses: device (agent) scope,
// so the data goes through, or around, the XCD-local L2 to the point where
// every XCD sees it, without an L2-wide write-back or invalidate.
constexpr int kDeviceCoherent = 16;   // SC1
constexpr int kBufferFormat = 0x00020000;   // raw 32-bit buffer descriptor word 3

struct Params {
  const char* q;
  const char* k;
  const char* v;
  const int32_t* ctx_lens;
  const int32_t* chunk_lens;
  float* out;
  float* lse;
  int* counters;    // [B*Hkv] arrival counters, zero between calls
  float* ws_o;      // [2*P][Rcap][D] normalised partial outputs
  float* ws_lse;    // [2*P][Rcap] partial log-sum-exp
  int ws_o_bytes, ws_lse_bytes;
  int B, Hq, Hkv, g, C_max, S_max;
  int Rcap;         // C_max * g
  int P;            // persistent workgroups
  float sl2;        // scale * log2(e)
};

template <bool BF16, int D>
struct Cfg {
  static constexpr int kElt = BF16 ? 2 : 4;
  static constexpr int kRowBytes = D * kElt;
  static constexpr int kChunks = kRowBytes / 16;          // 16-byte chunks per row
  static constexpr int kPitch = kRowBytes + 16;            // padded LDS row pitch
  static constexpr int kTileKeys = kTileBytes / kRowBytes;
  static constexpr int kLdsTile = kTileKeys * kPitch;      // LDS bytes of one staged tile
  static constexpr int kRowsPerPass = kThreads / kChunks;  // cache rows one block load covers
  static constexpr int kNSub = kTileKeys / kSub;
  static constexpr int kLoads = kTileBytes / (kThreads * 16);  // per thread, per tensor
  static constexpr int kQChunks = kChunks / 2;             // Q chunks held per lane
  static constexpr int kDC = D / 32;                       // 32-wide d blocks of O^T
};

// Byte offset of 16-byte chunk `c` of row `row` inside a staged LDS tile.  The
// 16-byte row padding shifts consecutive rows by four banks, so 16 lanes that
// read the same chunk of 16 consecutive rows hit 64 distinct banks.
template <class C>
__device__ __forceinline__ int lds_off(int row, int c) {
  return row * C::kPitch + 16 * c;
}

__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = (__bf16)lo;
  __bf16 b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
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
__device__ __forceinline__ int seq_c(uint32_t s) { return (int)(s & 0xffu); }
template <class C>
__device__ __forceinline__ int seq_tiles(uint32_t s) {
  return seq_c(s) == 0 ? 0 : (seq_T(s) + C::kTileKeys - 1) / C::kTileKeys;
}

// First tile of the contiguous tile range of persistent workgroup q.
__device__ __forceinline__ long long range_begin(long long q, long long N, int P) { return q * N / P; }
// Workgroup whose range holds global tile t.
__device__ __forceinline__ long long range_owner(long long t, long long N, int P) {
  return ((t + 1) * P - 1) / N;
}

template <bool BF16, int D>
__global__ __launch_bounds__(kThreads, 2) void verify_attn_kernel(Params p) {
  using C = Cfg<BF16, D>;
  __shared__ __attribute__((aligned(16))) char smem[2 * C::kLdsTile];
  __shared__ uint32_t seqs[kMaxSeqs];     // packed (T, c) of every sequence of the launch
  __shared__ int wave_sum[kWaves];
  __shared__ int start_pos[6];            // (b, kv head, tile) of this workgroup's first and last tile
  __shared__ int last_flag;
  char* ks = smem;
  char* vs = smem + C::kLdsTile;

  const int pid = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lr = lane & 31;     // row (or key, or d) index inside a 32-wide MFMA block
  const int half = lane >> 5;   // which half of the MFMA k dimension this lane feeds
  const int B = p.B, Hkv = p.Hkv, g = p.g;

  // ---- prologue: lengths into LDS; tiles per sequence; block-wide scan.
  // Thread tid owns the contiguous sequences [b_lo, b_hi).
  const int per = (B + kThreads - 1) / kThreads;
  const int b_lo = min(tid * per, B);
  const int b_hi = min(b_lo + per, B);
  int my_tiles = 0;
  for (int b = b_lo; b < b_hi; ++b) {
    const uint32_t s = load_seq(p, b);
    seqs[b] = s;
    my_tiles += seq_tiles<C>(s);
  }
  int incl = my_tiles;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wave_sum[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    before += w < wave ? wave_sum[w] : 0;
    total += wave_sum[w];
  }
  const long long N = (long long)total * Hkv;   // tiles of all units
  // Workgroups that get tiles: at most one per tile, so that every range is
  // non-empty and the pieces of a unit are exactly its owners pf..pl.
  const int Pe = (int)(N < p.P ? N : p.P);
  const long long g0 = pid < Pe ? range_begin(pid, N, Pe) : 0;
  const long long g1 = pid < Pe ? range_begin(pid + 1, N, Pe) : 0;
  // (b, kv head, tile) of this workgroup's first tile g0 and last tile g1-1,
  // found by the thread whose sequences hold them
  if (g0 < g1 && my_tiles > 0) {
    const long long base = (long long)(incl - my_tiles + before) * Hkv;   // tiles before b_lo
    const long long lim = base + (long long)my_tiles * Hkv;
#pragma unroll
    for (int w2 = 0; w2 < 2; ++w2) {
      const long long t = w2 == 0 ? g0 : g1 - 1;
      if (t < base || t >= lim) continue;
      long long pos = base;
      for (int b = b_lo; b < b_hi; ++b) {
        const int n = seq_tiles<C>(seqs[b]);
        const long long span = (long long)n * Hkv;
        if (t < pos + span) {
          const int off = (int)(t - pos);
          start_pos[3 * w2 + 0] = b;
          start_pos[3 * w2 + 1] = off / n;
          start_pos[3 * w2 + 2] = off % n;
          break;
        }
        pos += span;
      }
    }
  }
  __syncthreads();

  // ---- padding rows c_b <= i < C_max of the sequences b = pid (mod P):
  // out = 0, lse = -inf.
  for (int b = pid; b < B; b += p.P) {
    const int c = seq_c(seqs[b]);
    const int pad_rows = (p.C_max - c) * p.Hq;
    for (int idx = tid; idx < pad_rows * (D / 4); idx += kThreads) {
      const int r = idx / (D / 4);
      const int d4 = idx - r * (D / 4);
      const int i = c + r / p.Hq;
      const int h = r % p.Hq;
      const size_t orow = (size_t)(b * p.C_max + i) * p.Hq + h;
      *reinterpret_cast<f32x4*>(p.out + orow * D + 4 * d4) = f32x4{0.f, 0.f, 0.f, 0.f};
      if (d4 == 0) p.lse[orow] = -INFINITY;
    }
  }
  if (g0 >= g1) return;

  // ---- tile order.  The workgroup's range [g0, g1) starts inside a unit
  // shared with workgroup pid-1 (the first segment) and ends inside a unit
  // shared with pid+1 (the last segment), with whole units in between.  The
  // last segment is streamed first, then the range from g0 on: both pieces
  // of every shared unit are then done early in the launch, and the launch
  // ends on whole units, whose results need no merging.
  const int b0 = start_pos[0], kvh0 = start_pos[1], j0 = start_pos[2];
  const int b1 = start_pos[3], kvh1 = start_pos[4], j1 = start_pos[5];
  const long long s_last = g1 - 1 - j1;                  // first tile of the last tile's unit
  const bool rotated = s_last > g0 && j1 < seq_tiles<C>(seqs[b1]) - 1;
  const int count = (int)(g1 - g0);

  int cb = rotated ? b1 : b0, ckvh = rotated ? kvh1 : kvh0, cj = rotated ? 0 : j0;
  long long cg = rotated ? s_last : g0;                 // global index of the cursor's tile
  uint32_t cs = seqs[cb];
  int cn = seq_tiles<C>(cs);

  // prefetch registers: load j of thread tid takes row j*kRowsPerPass + r0 of
  // the tile, chunk c0; one wave instruction reads 1 KB of contiguous rows.
  const int r0 = tid / C::kChunks;
  const int c0 = tid % C::kChunks;
  u32x4 kreg[C::kLoads], vreg[C::kLoads];
  auto prefetch = [&](int b, int kvh, int j, uint32_t s, int n) {
    const int T = seq_T(s);
    const int hi = T - (n - 1 - j) * C::kTileKeys;
    const int lo = hi > C::kTileKeys ? hi - C::kTileKeys : 0;
    const int nk = hi - lo;
    // K/V slab of the unit; byte offsets inside it fit in 32 bits (host check)
    const size_t slab = ((size_t)b * Hkv + kvh) * (size_t)p.S_max * C::kRowBytes;
    const char* __restrict__ kp = p.k + slab;
    const char* __restrict__ vp = p.v + slab;
    const uint32_t base = (uint32_t)(lo + r0) * C::kRowBytes + 16u * c0;
#pragma unroll
    for (int j2 = 0; j2 < C::kLoads; ++j2) {
      const uint32_t off = base + (uint32_t)(j2 * C::kRowsPerPass * C::kRowBytes);
      if (j2 * C::kRowsPerPass + r0 < nk) {
        kreg[j2] = *reinterpret_cast<const u32x4*>(kp + off);
        vreg[j2] = *reinterpret_cast<const u32x4*>(vp + off);
      } else {
        kreg[j2] = u32x4{0u, 0u, 0u, 0u};
        vreg[j2] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto stage = [&]() {
    const int base = lds_off<C>(r0, c0);
#pragma unroll
    for (int j2 = 0; j2 < C::kLoads; ++j2) {
      const int off = base + j2 * C::kRowsPerPass * C::kPitch;
      *reinterpret_cast<u32x4*>(ks + off) = kreg[j2];
      *reinterpret_cast<u32x4*>(vs + off) = vreg[j2];
    }
  };

  // per-segment state
  u32x4 qreg[C::kQChunks];
  f32x16 o[C::kDC];
  float m_run = 0.f, l_run = 0.f;
  int n_rt4 = 1, n_kg = 1, rt = 0, kg = 0, R = 0, row = 0, tok = 0, vis = 0, l_ctx = 0;
  bool has_rows = false, row_valid = false;
  long long seg_g = g0;       // global index of the segment's first tile

  // Wave roles and Q operand of the unit (b, kvh) with packed lengths s.
  auto start_unit = [&](int b, int kvh, uint32_t s) {
    const int c = seq_c(s);
    R = c * g;
    l_ctx = seq_T(s) - c;
    const int n_rt = (R + kRowTile - 1) / kRowTile;
    n_rt4 = n_rt == 3 ? 4 : n_rt;
    n_kg = kWaves / n_rt4;
    rt = wave % n_rt4;
    kg = wave / n_rt4;
    has_rows = rt < n_rt;
    row = rt * kRowTile + lr;
    row_valid = has_rows && row < R;
    tok = row_valid ? row / g : 0;
    vis = row_valid ? l_ctx + tok : 0x7fffffff;   // last visible key of this lane's row
    const char* qrow = p.q + ((size_t)(b * p.C_max + tok) * p.Hq + kvh * g + (row_valid ? row % g : 0)) *
                                 C::kRowBytes;
#pragma unroll
    for (int j2 = 0; j2 < C::kQChunks; ++j2)
      qreg[j2] = row_valid ? *reinterpret_cast<const u32x4*>(qrow + 16 * (2 * j2 + half))
                           : u32x4{0u, 0u, 0u, 0u};
  };

  // Partial results go through raw buffer descriptors so that they can use
  // the device-coherent cache policy at 16-byte width.
  const __amdgpu_buffer_rsrc_t ws_o_rsrc = __builtin_amdgcn_make_buffer_rsrc(p.ws_o, 0, p.ws_o_bytes, kBufferFormat);
  const __amdgpu_buffer_rsrc_t ws_lse_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(p.ws_lse, 0, p.ws_lse_bytes, kBufferFormat);

  // Merge every published piece of a unit (run by the piece that arrives
  // last).  Piece q (pf <= q <= pl) sits in slot 2q, except the first one,
  // which is the last segment (slot 2q+1) of a workgroup whose range began
  // before the unit.
  auto merge_unit = [&](int unit, long long unit_first, int n_unit) {
    const long long pf = range_owner(unit_first, N, Pe);
    const long long pl = range_owner(unit_first + n_unit - 1, N, Pe);
    const int slot_first = (int)(2 * pf + (range_begin(pf, N, Pe) < unit_first ? 1 : 0));
    const int ub = unit / Hkv;
    const int ukvh = unit - ub * Hkv;
    const int uR = seq_c(seqs[ub]) * g;
    constexpr int kBatch = 4;
    for (int idx = tid; idx < uR * (D / 4); idx += kThreads) {
      const int r = idx / (D / 4);
      const int d0 = 4 * (idx - r * (D / 4));
      float m = -INFINITY, z = 0.f;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (long long q0 = pf; q0 <= pl; q0 += kBatch) {
        float lq[kBatch];
        f32x4 x[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const long long q = q0 + u;
          const int sl = q == pf ? slot_first : (int)(2 * q);
          const int srow = sl * p.Rcap + r;
          if (q <= pl) {
            lq[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ws_lse_rsrc, srow * 4, 0,
                                                                                 kDeviceCoherent));
            x[u] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                 ws_o_rsrc, (srow * D + d0) * 4, 0, kDeviceCoherent));
          }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          if (q0 + u > pl) break;
          const float nm = fmaxf(m, lq[u]);
          const float a = expf(m - nm);
          const float w = expf(lq[u] - nm);
          z = z * a + w;
          acc = acc * a + w * x[u];
          m = nm;
        }
      }
      const size_t orow = (size_t)(ub * p.C_max + r / g) * p.Hq + ukvh * g + r % g;
      *reinterpret_cast<f32x4*>(p.out + orow * D + d0) = acc * (1.f / z);
      if (d0 == 0) p.lse[orow] = m + logf(z);
    }
    if (tid == 0)   // ready for the next call
      __hip_atomic_store(p.counters + unit, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };

  // Publication of a partial piece is pipelined: its stores are issued at
  // the end of the segment; one iteration later, after the next tile's stage
  // has waited for memory anyway, the remaining stores are waited for and
  // the piece is counted; the count comes back during that tile's compute.
  bool pub_pending = false;     // a piece's stores are issued, not yet counted
  int pub_unit = 0, pub_n = 0;
  long long pub_first = 0;
  auto count_piece = [&]() -> int {
    const long long pf = range_owner(pub_first, N, Pe);
    const long long pl = range_owner(pub_first + pub_n - 1, N, Pe);
    int old = 0;
    if (tid == 0) old = __hip_atomic_fetch_add(p.counters + pub_unit, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return old == (int)(pl - pf) ? 1 : 0;
  };

  prefetch(cb, ckvh, cj, cs, cn);
  start_unit(cb, ckvh, cs);

  for (int v = 0; v < count; ++v) {
    const int b = cb, kvh = ckvh, j = cj, n = cn;
    const uint32_t s = cs;
    const long long gt = cg;
    const bool seg_first = gt == g0 || j == 0;
    const bool seg_last = gt == g1 - 1 || j == n - 1;

    // advance the cursor to the next tile in the workgroup's order
    if (v + 1 < count) {
      if (rotated && gt == g1 - 1) {
        cb = b0; ckvh = kvh0; cj = j0; cg = g0;
        cs = seqs[cb];
        cn = seq_tiles<C>(cs);
      } else {
        ++cg;
        if (++cj == cn) {
          cj = 0;
          if (++ckvh == Hkv) {
            ckvh = 0;
            do {
              ++cb;
            } while (seq_tiles<C>(seqs[cb]) == 0);   // in range: the next tile exists
            cs = seqs[cb];
            cn = seq_tiles<C>(cs);
          }
        }
      }
    }
    __syncthreads();   // every wave is done reading the previous tile
    stage();
    const bool publishing = pub_pending;
    if (publishing) {
      // the piece's device-coherent stores must be acknowledged before it
      // is counted; the compiler fences keep stores, wait and count in order
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      __builtin_amdgcn_s_waitcnt(0);
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
    }
    __syncthreads();
    const int is_last = publishing ? count_piece() : 0;
    if (v + 1 < count) prefetch(cb, ckvh, cj, cs, cn);

    const int T = seq_T(s);
    const int hi = T - (n - 1 - j) * C::kTileKeys;
    const int lo = hi > C::kTileKeys ? hi - C::kTileKeys : 0;
    const int nk = hi - lo;

    if (seg_first) {
      seg_g = gt;
#pragma unroll
      for (int dc = 0; dc < C::kDC; ++dc) o[dc] = f32x16{};
      m_run = -INFINITY;   // running row max, log2 units
      l_run = 0.f;         // running row sum of 2^(s - m_run)
    }

    if (has_rows) {
      for (int sub = kg; sub < C::kNSub; sub += n_kg) {
        if (sub * kSub >= nk) break;
        const int key0 = lo + sub * kSub;            // absolute index of the subtile's key 0
        const int krow = sub * kSub + lr;            // this lane's K row in the tile

        // S^T = K Q^T for 32 keys x 32 rows
        f32x16 sc = f32x16{};
#pragma unroll
        for (int j2 = 0; j2 < C::kQChunks; ++j2) {
          const u32x4 kop = *reinterpret_cast<const u32x4*>(ks + lds_off<C>(krow, 2 * j2 + half));
          if constexpr (BF16) {
            sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kop),
                                                         __builtin_bit_cast(bf16x8, qreg[j2]), sc, 0, 0, 0);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              sc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(kop[e]), __uint_as_float(qreg[j2][e]),
                                                        sc, 0, 0, 0);
          }
        }

        // scale, mask, online softmax; lane holds row `row`, keys
        // key0 + 8*(r/4) + 4*half + r%4 for r = 0..15
        const bool edge = (key0 + kSub > hi) || (key0 + kSub - 1 > l_ctx);
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float x = sc[r] * p.sl2;
          if (edge) {
            const int key = key0 + 8 * (r >> 2) + 4 * half + (r & 3);
            if (key >= hi || key > vis) x = -INFINITY;
          }
          sc[r] = x;
          mx = fmaxf(mx, x);
        }
        mx = fmaxf(mx, xor32(mx));
        const float m_new = fmaxf(m_run, mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
        float rs = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sc[r] = __builtin_amdgcn_exp2f(sc[r] - m_use);
          rs += sc[r];
        }
        rs += xor32(rs);
        l_run = l_run * alpha + rs;
        m_run = m_new;
#pragma unroll
        for (int dc = 0; dc < C::kDC; ++dc) o[dc] *= alpha;

        // O^T += V^T P^T
        if constexpr (BF16) {
          u32x4 pb[2];
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
            for (int w = 0; w < 4; ++w) pb[t2][w] = pack_bf16x2(sc[8 * t2 + 2 * w], sc[8 * t2 + 2 * w + 1]);
#pragma unroll
          for (int dc = 0; dc < C::kDC; ++dc) {
            const int d = dc * 32 + lr;
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
              // A operand: V[key(e)][d] for the 8 keys e of this lane's k half
              i16x8 vop;
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const int vrow = sub * kSub + 16 * t2 + 8 * (e >> 2) + 4 * half + (e & 3);
                vop[e] = *reinterpret_cast<const short*>(vs + lds_off<C>(vrow, d >> 3) + 2 * (d & 7));
              }
              o[dc] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vop),
                                                              __builtin_bit_cast(bf16x8, pb[t2]), o[dc], 0, 0, 0);
            }
            // keep the gathers of one 32-wide d block live at a time
            __builtin_amdgcn_sched_barrier(0);
          }
        } else {
#pragma unroll
          for (int dc = 0; dc < C::kDC; ++dc) {
            const int d = dc * 32 + lr;
#pragma unroll
            for (int u = 0; u < 16; ++u) {
              const int vrow = sub * kSub + 8 * (u >> 2) + 4 * half + (u & 3);
              const float x = *reinterpret_cast<const float*>(vs + lds_off<C>(vrow, d >> 2) + 4 * (d & 3));
              o[dc] = __builtin_amdgcn_mfma_f32_32x32x2f32(x, sc[u], o[dc], 0, 0, 0);
            }
          }
        }
      }
    }

    // the counted piece: the last one to arrive merges all of its unit's pieces
    if (publishing) {
      if (tid == 0) last_flag = is_last;
      __syncthreads();
      if (last_flag) merge_unit(pub_unit, pub_first, pub_n);
      pub_pending = false;
    }
    if (!seg_last) continue;

    // ---- end of a segment: merge the key groups of each row tile via LDS
    if (n_kg > 1) {
      __syncthreads();
      float* mbuf = reinterpret_cast<float*>(smem);
      constexpr int kRegion = 128 + C::kDC * 16 * 64;   // stats (2 x 64) then O
      if (kg > 0 && has_rows) {
        float* reg = mbuf + ((kg - 1) * n_rt4 + rt) * kRegion;
        reg[lane] = m_run;
        reg[64 + lane] = l_run;
#pragma unroll
        for (int dc = 0; dc < C::kDC; ++dc)
#pragma unroll
          for (int r = 0; r < 16; ++r) reg[128 + (dc * 16 + r) * 64 + lane] = o[dc][r];
      }
      __syncthreads();
      if (kg == 0 && has_rows) {
        float M = m_run;
        for (int k2 = 1; k2 < n_kg; ++k2) M = fmaxf(M, mbuf[((k2 - 1) * n_rt4 + rt) * kRegion + lane]);
        const float Muse = M == -INFINITY ? 0.f : M;
        const float a0 = __builtin_amdgcn_exp2f(m_run - Muse);
        l_run *= a0;
#pragma unroll
        for (int dc = 0; dc < C::kDC; ++dc) o[dc] *= a0;
        for (int k2 = 1; k2 < n_kg; ++k2) {
          const float* reg = mbuf + ((k2 - 1) * n_rt4 + rt) * kRegion;
          const float w = __builtin_amdgcn_exp2f(reg[lane] - Muse);
          l_run += reg[64 + lane] * w;
#pragma unroll
          for (int dc = 0; dc < C::kDC; ++dc)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[dc][r] += w * reg[128 + (dc * 16 + r) * 64 + lane];
        }
        m_run = M;
      }
    }

    // ---- write: the whole unit (final result) or this workgroup's piece
    // of it (partial).  Every valid row saw at least one key of the segment,
    // so l_run > 0.
    const long long unit_first = gt - j;                 // global index of the unit's tile 0
    const bool whole = seg_g == unit_first && j == n - 1;
    const int slot = 2 * pid + (seg_g == g0 ? 0 : 1);
    if (kg == 0 && row_valid) {
      const float inv = 1.f / l_run;
      const float lse_val = (m_run + log2f(l_run)) * kLn2;
      if (whole) {
        const size_t orow = (size_t)(b * p.C_max + tok) * p.Hq + kvh * g + row % g;
        float* dst = p.out + orow * D;
        if (half == 0) p.lse[orow] = lse_val;
#pragma unroll
        for (int dc = 0; dc < C::kDC; ++dc)
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = dc * 32 + 8 * g4 + 4 * half;
            *reinterpret_cast<f32x4*>(dst + d0) = f32x4{o[dc][4 * g4] * inv, o[dc][4 * g4 + 1] * inv,
                                                        o[dc][4 * g4 + 2] * inv, o[dc][4 * g4 + 3] * inv};
          }
      } else {
        // read by another workgroup, possibly on another XCD: device-coherent stores
        const int srow = slot * p.Rcap + row;
        if (half == 0)
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, lse_val), ws_lse_rsrc, srow * 4, 0,
                                                kDeviceCoherent);
#pragma unroll
        for (int dc = 0; dc < C::kDC; ++dc)
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = dc * 32 + 8 * g4 + 4 * half;
            const f32x4 val = {o[dc][4 * g4] * inv, o[dc][4 * g4 + 1] * inv, o[dc][4 * g4 + 2] * inv,
                               o[dc][4 * g4 + 3] * inv};
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, val), ws_o_rsrc, (srow * D + d0) * 4,
                                                   0, kDeviceCoherent);
          }
      }
    }
    if (!whole) {
      pub_pending = true;
      pub_unit = b * Hkv + kvh;
      pub_first = unit_first;
      pub_n = n;
    }
    // the next tile starts a new unit: load its Q now, so that it arrives
    // while this workgroup waits for the next tile anyway
    if (v + 1 < count) start_unit(cb, ckvh, cs);
  }

  // ---- a piece from the last tile is still to be counted
  if (pub_pending) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __syncthreads();
    const int is_last = count_piece();
    if (tid == 0) last_flag = is_last;
    __syncthreads();
    if (last_flag) merge_unit(pub_unit, pub_first, pub_n);
  }
}

// Zero the arrival counters at the start of a workspace.
__global__ void zero_counters_kernel(int* counters, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) counters[i] = 0;
}

// ---------------------------------------------------------------- host side

int key_tile(int dtype, int D) {
  const int elt = dtype == SPECMOE_BF16 ? 2 : 4;
  return kTileBytes / (D * elt);
}

struct Plan {
  int g, P, Rcap, seqs_per_launch;
  size_t counter_bytes, ws_lse_off, ws_o_off, ws_bytes;
};

int validate_desc(const specmoe_verify_desc* d) {
  if (!d) return SPECMOE_ERR_NULL_POINTER;
  if (d->dtype != SPECMOE_F32 && d->dtype != SPECMOE_BF16) return SPECMOE_ERR_DTYPE;
  if (d->D != 64 && d->D != 128) return SPECMOE_ERR_HEAD_DIM;
  if (d->B < 0 || d->Hq <= 0 || d->Hkv <= 0 || d->C_max < 1 || d->S_max < d->C_max)
    return SPECMOE_ERR_SHAPE;
  if (d->Hq % d->Hkv != 0) return SPECMOE_ERR_GQA;
  const int64_t g = d->Hq / d->Hkv;
  if ((int64_t)d->C_max * g > kMaxRows) return SPECMOE_ERR_ROWS;
  if (d->grid_blocks < 0 || d->grid_blocks > (1 << 20)) return SPECMOE_ERR_GRID;
  // partial results are addressed through 32-bit buffer descriptors
  const int64_t grid = d->grid_blocks ? d->grid_blocks : kDefaultGrid;
  if (2 * grid * (int64_t)d->C_max * g * d->D * 4 >= ((int64_t)1 << 31)) return SPECMOE_ERR_GRID;
  // index arithmetic: (sequence, token, head) row indices stay in 32 bits,
  // byte offsets inside one (sequence, KV head) slab are 32-bit, packed
  // sequence lengths need T < 2^24, tile counts per launch stay in 32 bits.
  if ((int64_t)d->B * d->C_max * d->Hq >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  const int64_t elt = d->dtype == SPECMOE_BF16 ? 2 : 4;
  if ((int64_t)d->S_max * d->D * elt >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  if (d->S_max >= (1 << 24)) return SPECMOE_ERR_SHAPE;
  const int64_t tile = key_tile(d->dtype, d->D);
  if ((int64_t)kMaxSeqs * d->Hkv * ((d->S_max + tile - 1) / tile) >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  return SPECMOE_OK;
}

Plan make_plan(const specmoe_verify_desc* d) {
  Plan pl;
  pl.g = d->Hq / d->Hkv;
  pl.P = d->grid_blocks ? d->grid_blocks : kDefaultGrid;
  pl.Rcap = d->C_max * pl.g;
  pl.seqs_per_launch = d->B < kMaxSeqs ? d->B : kMaxSeqs;
  const size_t units = (size_t)pl.seqs_per_launch * d->Hkv;
  pl.counter_bytes = (units * sizeof(int) + 255) / 256 * 256;
  const size_t slots = (size_t)2 * pl.P * pl.Rcap;
  pl.ws_lse_off = pl.counter_bytes;
  pl.ws_o_off = pl.ws_lse_off + (slots * sizeof(float) + 255) / 256 * 256;
  pl.ws_bytes = pl.ws_o_off + slots * d->D * sizeof(float);
  return pl;
}

template <bool BF16, int D>
void launch(Params p, const Plan& pl, hipStream_t stream, const specmoe_verify_desc* d) {
  using C = Cfg<BF16, D>;
  const int B = p.B;
  if (d->ev_main_begin) (void)hipEventRecord(static_cast<hipEvent_t>(d->ev_main_begin), stream);
  // batches beyond kMaxSeqs sequences run as consecutive launches on the stream
  for (int b0 = 0; b0 < B; b0 += kMaxSeqs) {
    Params s = p;
    s.B = B - b0 < kMaxSeqs ? B - b0 : kMaxSeqs;
    s.q = p.q + (size_t)b0 * p.C_max * p.Hq * C::kRowBytes;
    const size_t slab = (size_t)b0 * p.Hkv * p.S_max * C::kRowBytes;
    s.k = p.k + slab;
    s.v = p.v + slab;
    s.ctx_lens = p.ctx_lens + b0;
    s.chunk_lens = p.chunk_lens + b0;
    s.out = p.out + (size_t)b0 * p.C_max * p.Hq * D;
    s.lse = p.lse + (size_t)b0 * p.C_max * p.Hq;
    hipLaunchKernelGGL((verify_attn_kernel<BF16, D>), dim3(pl.P), dim3(kThreads), 0, stream, s);
  }
  if (d->ev_main_end) (void)hipEventRecord(static_cast<hipEvent_t>(d->ev_main_end), stream);
}

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

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
  const int n = (int)(pl.counter_bytes / sizeof(int));
  (void)hipGetLastError();
  hipLaunchKernelGGL(zero_counters_kernel, dim3((n + 255) / 256), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<int*>(workspace), n);
  return hipGetLastError() == hipSuccess ? SPECMOE_OK : SPECMOE_ERR_LAUNCH;
}

int32_t specmoe_verify_attn_key_tile(const specmoe_verify_desc* desc) {
  if (!desc) return SPECMOE_ERR_NULL_POINTER;
  if (desc->dtype != SPECMOE_F32 && desc->dtype != SPECMOE_BF16) return SPECMOE_ERR_DTYPE;
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
    case SPECMOE_ERR_GRID: return "grid_blocks must be 0 (default) or in [1, 2^20], with partial results under 2 GB";
    case SPECMOE_ERR_WORKSPACE: return "workspace too small";
    case SPECMOE_ERR_ALIGN: return "q, k_cache, v_cache, out and workspace must be 16-byte aligned";
    case SPECMOE_ERR_SCALE: return "scale is not finite";
    case SPECMOE_ERR_LAUNCH: return "HIP kernel launch failed";
    default: return "unknown status";
  }
}

int specmoe_verify_attn(const void* q, const void* k_cache, const void* v_cache, const int32_t* ctx_lens,
                        const int32_t* chunk_lens, float scale, float* out, float* lse, void* stream,
                        const specmoe_verify_desc* desc) {
  const int st = validate_desc(desc);
  if (st != SPECMOE_OK) return st;
  if (desc->B == 0) return SPECMOE_OK;   // nothing to read or write
  if (!q || !k_cache || !v_cache || !ctx_lens || !chunk_lens || !out || !lse) return SPECMOE_ERR_NULL_POINTER;
  if (!isfinite(scale)) return SPECMOE_ERR_SCALE;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out)) return SPECMOE_ERR_ALIGN;
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
  char* ws = static_cast<char*>(desc->workspace);
  p.counters = reinterpret_cast<int*>(ws);
  p.ws_lse = reinterpret_cast<float*>(ws + pl.ws_lse_off);
  p.ws_o = reinterpret_cast<float*>(ws + pl.ws_o_off);
  p.ws_o_bytes = (int)(pl.ws_bytes - pl.ws_o_off);
  p.ws_lse_bytes = (int)(pl.ws_o_off - pl.ws_lse_off);
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
  const bool bf16 = desc->dtype == SPECMOE_BF16;
  if (bf16 && desc->D == 128) launch<true, 128>(p, pl, s, desc);
  else if (bf16) launch<true, 64>(p, pl, s, desc);
  else if (desc->D == 128) launch<false, 128>(p, pl, s, desc);
  else launch<false, 64>(p, pl, s, desc);
  if (hipGetLastError() != hipSuccess) return SPECMOE_ERR_LAUNCH;
  return SPECMOE_OK;
}

}  // extern "C"
