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
constexpr int kTileBytes = 16384;    // K bytes (and V bytes) of one tile
constexpr int kDefaultGrid = 512;    // persistent workgroups: 2 per CU on MI355X's 256 CUs
constexpr int kMaxSeqs = 1024;       // sequences per launch (their lengths live in LDS)
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
  int* counters;    // [B*Hkv] per-unit tile counts of published pieces, zero between calls
  int* claims;      // [P][4] tail-chunk claim marks
  int* thief_ctr;   // steal probes of the current call, zero between calls
  int* gen;         // generation: a call's claim/piece mark is gen + 1
  float* ws_o;      // [slots][Rcap][D] normalised partial outputs
  float* ws_lse;    // [slots][Rcap] partial log-sum-exp
  int* ws_tag;      // [slots][2] (mark, unit) of the piece in each slot
  int ws_o_bytes, ws_lse_bytes, ws_tag_bytes;
  int deterministic;  // no stealing
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
  static constexpr int kSlots = kChunks + 1;               // LDS slots per row: the chunks + one pad
  static constexpr int kPitch = 16 * kSlots;               // padded LDS row pitch
  static constexpr int kTileKeys = kTileBytes / kRowBytes;
  static constexpr int kLdsTile = kTileKeys * kPitch;      // LDS bytes of one staged K (or V) tile
  static constexpr int kInst = (kTileKeys * kSlots + 63) / 64;   // 64-slot DMA instructions per tile
  static constexpr int kNSub = kTileKeys / kSub;
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

// Tile schedule shared by every workgroup of a launch.  The tiles of all
// units form one list [0, N) cut into Pe equal contiguous home ranges (one
// per workgroup).  The last ~quarter of each range is cut into nt tail
// chunks of cs tiles that other workgroups may steal; the rest is the head.
struct Sched {
  int N, Pe, nt, cs;
  __device__ int range_begin(int q) const { return (int)((long long)q * N / Pe); }
  // home range holding tile t
  __device__ int range_owner(int t) const { return (int)(((long long)(t + 1) * Pe - 1) / N); }
  __device__ int head_end(int q) const { return range_begin(q + 1) - nt * cs; }
  // sub-range x of range q: x = 0 is the head, x = 1 + i tail chunk i
  __device__ int sub_begin(int q, int x) const { return x == 0 ? range_begin(q) : head_end(q) + (x - 1) * cs; }
  __device__ int sub_end(int q, int x) const { return x == 0 ? head_end(q) : head_end(q) + x * cs; }
  __device__ int sub_index(int t) const {
    const int q = range_owner(t);
    const int h = head_end(q);
    return q * (nt + 1) + (t < h ? 0 : 1 + (t - h) / cs);
  }
};

// Merge every published piece of a unit; run by all threads of the
// workgroup whose piece completed the unit's tile count.  A piece sits in
// slot 2*x + side of the sub-range x where it starts and is tagged
// (mark, unit); the candidates are both slots of every sub-range that meets
// the unit, taken in a fixed order.  Inlined: a call would make the
// streaming loop keep its live registers across the call boundary.
template <int D>
__device__ __forceinline__ void merge_unit(const Params& p, const Sched& sc, const uint32_t* seqs, char* lds,
                                        int mark, int unit, int unit_first, int n_unit) {
  const int tid = threadIdx.x;
  const int g = p.g, Hkv = p.Hkv;
  const __amdgpu_buffer_rsrc_t ws_o_rsrc = __builtin_amdgcn_make_buffer_rsrc(p.ws_o, 0, p.ws_o_bytes, kBufferFormat);
  const __amdgpu_buffer_rsrc_t ws_lse_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(p.ws_lse, 0, p.ws_lse_bytes, kBufferFormat);
  const __amdgpu_buffer_rsrc_t ws_tag_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(p.ws_tag, 0, p.ws_tag_bytes, kBufferFormat);
  const int unit_last = unit_first + n_unit - 1;
  const int qf = sc.range_owner(unit_first);
  const int ql = sc.range_owner(unit_last);
  const int per_q = 2 * (sc.nt + 1);
  const int ncand = (ql - qf + 1) * per_q;
  unsigned char* valid = reinterpret_cast<unsigned char*>(lds);
  __syncthreads();   // the LDS tile is free: every wave is past its compute
  for (int c = tid; c < ncand; c += kThreads) {
    const int q = qf + c / per_q;
    const int x = (c % per_q) >> 1;
    const int slot = 2 * (q * (sc.nt + 1) + x) + (c & 1);
    bool ok = sc.sub_begin(q, x) <= unit_last && sc.sub_end(q, x) > unit_first;
    if (ok) {
      const int tm = __builtin_amdgcn_raw_buffer_load_b32(ws_tag_rsrc, slot * 8, 0, kDeviceCoherent);
      const int tu = __builtin_amdgcn_raw_buffer_load_b32(ws_tag_rsrc, slot * 8 + 4, 0, kDeviceCoherent);
      ok = tm == mark && tu == unit;
    }
    valid[c] = ok ? 1 : 0;
  }
  __syncthreads();
  const int ub = unit / Hkv;
  const int ukvh = unit - ub * Hkv;
  const int uR = seq_c(seqs[ub]) * g;
  constexpr int kBatch = 4;
  for (int idx = tid; idx < uR * (D / 4); idx += kThreads) {
    const int r = idx / (D / 4);
    const int d0 = 4 * (idx - r * (D / 4));
    float m = -INFINITY, z = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    int c = 0;
    while (c < ncand) {
      float lq[kBatch];
      f32x4 xv[kBatch];
      int got = 0;
      // gather up to kBatch valid pieces, then fold them in
      for (; c < ncand && got < kBatch; ++c) {
        if (!valid[c]) continue;
        const int q = qf + c / per_q;
        const int x = (c % per_q) >> 1;
        const int srow = (2 * (q * (sc.nt + 1) + x) + (c & 1)) * p.Rcap + r;
        lq[got] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ws_lse_rsrc, srow * 4, 0,
                                                                                kDeviceCoherent));
        xv[got] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                ws_o_rsrc, (srow * D + d0) * 4, 0, kDeviceCoherent));
        ++got;
      }
      for (int u = 0; u < got; ++u) {
        const float nm = fmaxf(m, lq[u]);
        const float a = expf(m - nm);
        const float w = expf(lq[u] - nm);
        z = z * a + w;
        acc = acc * a + w * xv[u];
        m = nm;
      }
    }
    const size_t orow = (size_t)(ub * p.C_max + r / g) * p.Hq + ukvh * g + r % g;
    *reinterpret_cast<f32x4*>(p.out + orow * D + d0) = acc * (1.f / z);
    if (d0 == 0) p.lse[orow] = m + logf(z);
  }
  if (tid == 0)   // ready for the next call
    __hip_atomic_store(p.counters + unit, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <bool BF16, int D>
__global__ __launch_bounds__(kThreads, 2) void verify_attn_kernel(Params p) {
  using C = Cfg<BF16, D>;
  // two tile buffers, each a K tile followed by a V tile
  __shared__ __attribute__((aligned(16))) char smem[2 * 2 * C::kLdsTile];
  __shared__ uint32_t seqs[kMaxSeqs];     // packed (T, c) of every sequence of the launch
  __shared__ int pref[kMaxSeqs + 1];      // tiles per KV head of the sequences before b
  __shared__ int wave_sum[kWaves];
  __shared__ int sh_int[4];               // broadcast slots: mark, claim result, flag, probe result

  const int pid = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lr = lane & 31;     // row (or key, or d) index inside a 32-wide MFMA block
  const int half = lane >> 5;   // which half of the MFMA k dimension this lane feeds
  const int B = p.B, Hkv = p.Hkv, g = p.g;

  // ---- prologue: lengths and tile prefix sums into LDS (block-wide scan).
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
  if (tid == 0) sh_int[0] = 1 + __hip_atomic_load(p.gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    before += w < wave ? wave_sum[w] : 0;
    total += wave_sum[w];
  }
  {
    int run = incl - my_tiles + before;
    for (int b = b_lo; b < b_hi; ++b) {
      pref[b] = run;
      run += seq_tiles<C>(seqs[b]);
    }
    if (tid == kThreads - 1) pref[B] = total;
  }
  const int mark = sh_int[0];   // this call's claim / piece mark (generation + 1)
  Sched sc;
  sc.N = total * Hkv;           // tiles of all units (< 2^31, host check)
  // workgroups that get tiles: at most one per tile, so no home range is empty
  sc.Pe = sc.N < p.P ? sc.N : p.P;
  {
    const int S = sc.Pe > 0 ? sc.N / sc.Pe : 0;
    if (p.deterministic || S < 8) {
      sc.nt = 0;
      sc.cs = 1;
    } else {
      // chunks of at least 2 tiles: the owner claims a chunk two tiles
      // before it would stream it, so the claim is settled in time
      const int tail = S / 4;
      sc.cs = max(2, (tail + 3) / 4);
      sc.nt = min(4, tail / sc.cs);
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
  if (pid >= sc.Pe) return;

  // (b, kv head, tile) of global tile t: a 64-ary search of the prefix sums
  // done by every wave on its own (two LDS reads and two ballots).
  auto locate = [&](int t, int& ob, int& okvh, int& oj) {
    const int tq = t / Hkv;                      // tiles per KV head before t's sequence, at most
    const int step = (B + 64) / 64;              // B + 1 prefix entries in 64 groups
    const int i1 = min(lane * step, B);
    const unsigned long long m1 = __ballot(pref[i1] <= tq);
    const int base = (63 - __builtin_clzll(m1)) * step;
    const int i2 = min(base + lane, B);
    const unsigned long long m2 = __ballot(lane < step && pref[i2] <= tq);
    const int b = base + 63 - __builtin_clzll(m2);
    const int n = seq_tiles<C>(seqs[b]);
    const int off = t - Hkv * pref[b];
    ob = b;
    okvh = off / n;
    oj = off - okvh * n;
  };

  // K/V tile (b, kvh, j) straight from HBM into LDS buffer `buf`.  Each
  // 64-lane DMA instruction fills 64 consecutive 16-byte LDS slots, i.e.
  // 1 KB of consecutive cache rows with their pad slots; a pad lane re-reads
  // a chunk of its own row and rows past the end of a partial tile re-read
  // the tile's last row, so every slot holds finite data from the same
  // cache lines.  Wave w issues instructions w, w + 4, ...
  auto dma_tile = [&](int buf, int b, int kvh, int j, uint32_t s, int n) {
    const int T = seq_T(s);
    const int hi = T - (n - 1 - j) * C::kTileKeys;
    const int lo = hi > C::kTileKeys ? hi - C::kTileKeys : 0;
    const int last = hi - lo - 1;
    // K/V slab of the unit; byte offsets inside it fit in 32 bits (host check)
    const size_t slab = ((size_t)b * Hkv + kvh) * (size_t)p.S_max * C::kRowBytes;
    const char* kp = p.k + slab + (size_t)lo * C::kRowBytes;
    const char* vp = p.v + slab + (size_t)lo * C::kRowBytes;
    char* kl = smem + buf * 2 * C::kLdsTile;
    char* vl = kl + C::kLdsTile;
#pragma unroll
    for (int i = wave; i < C::kInst; i += kWaves) {
      const int sl = 64 * i + lane;
      const int row = sl / C::kSlots;
      const int ch = sl - row * C::kSlots;
      const uint32_t off = (uint32_t)min(row, last) * C::kRowBytes + 16u * min(ch, C::kChunks - 1);
      if (sl < C::kTileKeys * C::kSlots) {
        __builtin_amdgcn_global_load_lds(kp + off, (__attribute__((address_space(3))) void*)(kl + 1024 * i), 16, 0, 0);
        __builtin_amdgcn_global_load_lds(vp + off, (__attribute__((address_space(3))) void*)(vl + 1024 * i), 16, 0, 0);
      }
    }
  };

  // per-segment state
  u32x4 qreg[C::kQChunks];
  f32x16 o[C::kDC];
  float m_run = 0.f, l_run = 0.f;
  int n_rt4 = 1, n_kg = 1, n_dh = 1, rt = 0, kg = 0, dh = 0, R = 0, row = 0, tok = 0, vis = 0, l_ctx = 0;
  bool has_rows = false, row_valid = false;

  // Wave roles and Q operand of the unit (b, kvh) with packed lengths s.
  // The 4 waves split into row tiles x key groups x halves of D.
  auto start_unit = [&](int b, int kvh, uint32_t s) {
    const int c = seq_c(s);
    R = c * g;
    l_ctx = seq_T(s) - c;
    const int n_rt = (R + kRowTile - 1) / kRowTile;
    n_rt4 = n_rt == 3 ? 4 : n_rt;
    n_kg = min(kWaves / n_rt4, C::kNSub);
    n_dh = kWaves / (n_rt4 * n_kg);
    rt = wave % n_rt4;
    kg = (wave / n_rt4) % n_kg;
    dh = wave / (n_rt4 * n_kg);
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
  const __amdgpu_buffer_rsrc_t ws_tag_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(p.ws_tag, 0, p.ws_tag_bytes, kBufferFormat);

  // Publication of a piece: its device-coherent stores are issued at the end
  // of its segment; the wait for every outstanding memory operation at the
  // top of the next tile covers them, and the piece's tiles are then added to
  // its unit's count.  The count comes back during that tile's compute; the
  // piece that completes the count merges the unit.
  bool pub_pending = false;
  int pub_unit = 0, pub_first = 0, pub_n = 0, pub_tiles = 0;
  auto count_piece = [&]() -> int {
    int old = 0;
    if (tid == 0)
      old = __hip_atomic_fetch_add(p.counters + pub_unit, pub_tiles, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return old + pub_tiles == pub_n ? 1 : 0;
  };
  // wait for every outstanding vector-memory operation of this thread (tile
  // DMA, Q loads, piece stores); the compiler fences keep it in place
  auto wait_all = [&]() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };

  // Claim tail chunk i of home range q for this call (owner or thief).
  auto claim = [&](int q, int i) -> int {
    const int old = __hip_atomic_fetch_max(p.claims + q * 4 + i, mark, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return old < mark ? 1 : 0;
  };

  // ---- runs: the head of the home range, extended by the owner's tail
  // chunks as long as it wins their claims; then stolen chunks.
  const int g0 = sc.range_begin(pid);
  const int h0 = sc.head_end(pid);
  int run_a = g0, run_e = h0;
  bool owner = true;
  int ext = 0;        // tail chunks added to the owner's run
  int issued = 0;     // tail-chunk claims issued by the owner
  int claim_tile = sc.nt > 0 ? max(g0, h0 - 2) : -1;   // tile during which claim `issued` goes out
  int claim_res = 0;
  if (sc.nt > 0 && h0 - 2 < g0) {
    // a one-tile head: claim chunk 0 before streaming
    if (tid == 0) sh_int[1] = claim(pid, 0);
    issued = 1;
    claim_tile = -1;
  }

  for (;;) {
    int cb, ckvh, cj;
    locate(run_a, cb, ckvh, cj);
    uint32_t cs = seqs[cb];
    int cn = seq_tiles<C>(cs);
    __syncthreads();           // both tile buffers are free
    dma_tile(0, cb, ckvh, cj, cs, cn);
    start_unit(cb, ckvh, cs);
    int seg_g = run_a;
    int buf = 0;

    for (int gt = run_a; gt < run_e; ++gt, buf ^= 1) {
      const int b = cb, kvh = ckvh, j = cj, n = cn;
      const uint32_t s = cs;
      wait_all();        // this tile's DMA (and the previous piece's stores) are done
      __syncthreads();   // ... for every wave; every wave is done with the other buffer
      // the owner's run grows by the next tail chunk if its claim was won
      if (owner && gt == run_e - 1 && ext < issued) {
        if (sh_int[1]) {
          run_e += sc.cs;
          ++ext;
          claim_tile = ext < sc.nt ? max(gt + 1, sc.head_end(pid) + ext * sc.cs - 2) : -1;
        } else {
          claim_tile = -1;
        }
      }
      const bool seg_first = gt == run_a || j == 0;
      const bool seg_last = gt == run_e - 1 || j == n - 1;
      const bool publishing = pub_pending;
      const int is_last = publishing ? count_piece() : 0;
      const bool claiming = owner && gt == claim_tile && issued < sc.nt;
      if (claiming && tid == 0) claim_res = claim(pid, issued);
      if (claiming) ++issued;
      if (gt + 1 < run_e) {
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
        dma_tile(buf ^ 1, cb, ckvh, cj, cs, cn);
      }

      const char* ks = smem + buf * 2 * C::kLdsTile;
      const char* vs = ks + C::kLdsTile;
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
        const int dc_lo = dh * (C::kDC / n_dh);
        const int dc_hi = dc_lo + C::kDC / n_dh;
        for (int sub = kg; sub < C::kNSub; sub += n_kg) {
          if (sub * kSub >= nk) break;
          const int key0 = lo + sub * kSub;            // absolute index of the subtile's key 0
          const int krow = sub * kSub + lr;            // this lane's K row in the tile

          // S^T = K Q^T for 32 keys x 32 rows
          f32x16 sacc = f32x16{};
#pragma unroll
          for (int j2 = 0; j2 < C::kQChunks; ++j2) {
            const u32x4 kop = *reinterpret_cast<const u32x4*>(ks + lds_off<C>(krow, 2 * j2 + half));
            if constexpr (BF16) {
              sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kop),
                                                             __builtin_bit_cast(bf16x8, qreg[j2]), sacc, 0, 0, 0);
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                sacc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(kop[e]),
                                                            __uint_as_float(qreg[j2][e]), sacc, 0, 0, 0);
            }
          }

          // scale, mask, online softmax; lane holds row `row`, keys
          // key0 + 8*(r/4) + 4*half + r%4 for r = 0..15
          const bool edge = (key0 + kSub > hi) || (key0 + kSub - 1 > l_ctx);
          float mx = -INFINITY;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            float x = sacc[r] * p.sl2;
            if (edge) {
              const int key = key0 + 8 * (r >> 2) + 4 * half + (r & 3);
              if (key >= hi || key > vis) x = -INFINITY;
            }
            sacc[r] = x;
            mx = fmaxf(mx, x);
          }
          mx = fmaxf(mx, xor32(mx));
          const float m_new = fmaxf(m_run, mx);
          const float m_use = m_new == -INFINITY ? 0.f : m_new;
          const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
          float rs = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            sacc[r] = __builtin_amdgcn_exp2f(sacc[r] - m_use);
            rs += sacc[r];
          }
          rs += xor32(rs);
          l_run = l_run * alpha + rs;
          m_run = m_new;
#pragma unroll
          for (int dc = 0; dc < C::kDC; ++dc)
            if (dc >= dc_lo && dc < dc_hi) o[dc] *= alpha;

          // O^T += V^T P^T for this wave's d blocks
          if constexpr (BF16) {
            u32x4 pb[2];
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
              for (int w = 0; w < 4; ++w)
                pb[t2][w] = pack_bf16x2(sacc[8 * t2 + 2 * w], sacc[8 * t2 + 2 * w + 1]);
#pragma unroll
            for (int dc = 0; dc < C::kDC; ++dc) {
              if (dc < dc_lo || dc >= dc_hi) continue;
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
              if (dc < dc_lo || dc >= dc_hi) continue;
              const int d = dc * 32 + lr;
#pragma unroll
              for (int u = 0; u < 16; ++u) {
                const int vrow = sub * kSub + 8 * (u >> 2) + 4 * half + (u & 3);
                const float x = *reinterpret_cast<const float*>(vs + lds_off<C>(vrow, d >> 2) + 4 * (d & 3));
                o[dc] = __builtin_amdgcn_mfma_f32_32x32x2f32(x, sacc[u], o[dc], 0, 0, 0);
              }
            }
          }
        }
      }

      // scratch space for merges: this tile's buffer, which every wave is
      // done reading after the merges' first barrier (the next DMA goes to
      // the other buffer)
      char* scratch = smem + buf * 2 * C::kLdsTile;

      // the counted piece: the one that completes its unit merges it
      if (publishing) {
        if (tid == 0) sh_int[2] = is_last;
        __syncthreads();
        if (sh_int[2]) merge_unit<D>(p, sc, seqs, scratch, mark, pub_unit, pub_first, pub_n);
        pub_pending = false;
      }
      // the owner's claim result, for the next tile's run extension
      if (claiming && tid == 0) sh_int[1] = claim_res;
      if (!seg_last) continue;

      // ---- end of a segment: merge the key groups of each (row tile, d
      // half) through LDS
      const int dc_lo = dh * (C::kDC / n_dh);
      const int dc_hi = dc_lo + C::kDC / n_dh;
      if (n_kg > 1) {
        __syncthreads();
        float* mbuf = reinterpret_cast<float*>(scratch);
        constexpr int kRegion = 128 + C::kDC * 16 * 64;   // stats (2 x 64) then O
        const int region = ((kg - 1) * n_rt4 + rt) * n_dh + dh;
        if (kg > 0 && has_rows) {
          float* reg = mbuf + region * kRegion;
          reg[lane] = m_run;
          reg[64 + lane] = l_run;
#pragma unroll
          for (int dc = 0; dc < C::kDC; ++dc)
            if (dc >= dc_lo && dc < dc_hi)
#pragma unroll
              for (int r = 0; r < 16; ++r) reg[128 + ((dc - dc_lo) * 16 + r) * 64 + lane] = o[dc][r];
        }
        __syncthreads();
        if (kg == 0 && has_rows) {
          float M = m_run;
          for (int k2 = 1; k2 < n_kg; ++k2)
            M = fmaxf(M, mbuf[(((k2 - 1) * n_rt4 + rt) * n_dh + dh) * kRegion + lane]);
          const float Muse = M == -INFINITY ? 0.f : M;
          const float a0 = __builtin_amdgcn_exp2f(m_run - Muse);
          l_run *= a0;
#pragma unroll
          for (int dc = 0; dc < C::kDC; ++dc) o[dc] *= a0;
          for (int k2 = 1; k2 < n_kg; ++k2) {
            const float* reg = mbuf + (((k2 - 1) * n_rt4 + rt) * n_dh + dh) * kRegion;
            const float w = __builtin_amdgcn_exp2f(reg[lane] - Muse);
            l_run += reg[64 + lane] * w;
#pragma unroll
            for (int dc = 0; dc < C::kDC; ++dc)
              if (dc >= dc_lo && dc < dc_hi)
#pragma unroll
                for (int r = 0; r < 16; ++r) o[dc][r] += w * reg[128 + ((dc - dc_lo) * 16 + r) * 64 + lane];
          }
          m_run = M;
        }
      }

      // ---- write: the whole unit (final result) or a piece of it.  Every
      // valid row saw at least one key of the segment, so l_run > 0.
      const int unit_first = gt - j;                 // global index of the unit's tile 0
      const bool whole = seg_g == unit_first && j == n - 1;
      const bool first_of_run = seg_g == run_a;
      const int slot = 2 * sc.sub_index(first_of_run ? run_a : seg_g) + (first_of_run ? 0 : 1);
      const int unit = b * Hkv + kvh;
      if (kg == 0 && row_valid) {
        const float inv = 1.f / l_run;
        const float lse_val = (m_run + log2f(l_run)) * kLn2;
        if (whole) {
          const size_t orow = (size_t)(b * p.C_max + tok) * p.Hq + kvh * g + row % g;
          float* dst = p.out + orow * D;
          if (half == 0 && dh == 0) p.lse[orow] = lse_val;
#pragma unroll
          for (int dc = 0; dc < C::kDC; ++dc)
            if (dc >= dc_lo && dc < dc_hi)
#pragma unroll
              for (int g4 = 0; g4 < 4; ++g4) {
                const int d0 = dc * 32 + 8 * g4 + 4 * half;
                *reinterpret_cast<f32x4*>(dst + d0) = f32x4{o[dc][4 * g4] * inv, o[dc][4 * g4 + 1] * inv,
                                                            o[dc][4 * g4 + 2] * inv, o[dc][4 * g4 + 3] * inv};
              }
        } else {
          // read by another workgroup, possibly on another XCD: device-coherent stores
          const int srow = slot * p.Rcap + row;
          if (half == 0 && dh == 0)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, lse_val), ws_lse_rsrc, srow * 4, 0,
                                                  kDeviceCoherent);
#pragma unroll
          for (int dc = 0; dc < C::kDC; ++dc)
            if (dc >= dc_lo && dc < dc_hi)
#pragma unroll
              for (int g4 = 0; g4 < 4; ++g4) {
                const int d0 = dc * 32 + 8 * g4 + 4 * half;
                const f32x4 val = {o[dc][4 * g4] * inv, o[dc][4 * g4 + 1] * inv, o[dc][4 * g4 + 2] * inv,
                                   o[dc][4 * g4 + 3] * inv};
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, val), ws_o_rsrc,
                                                       (srow * D + d0) * 4, 0, kDeviceCoherent);
              }
        }
      }
      if (!whole) {
        if (tid == 0) {
          __builtin_amdgcn_raw_buffer_store_b32(mark, ws_tag_rsrc, slot * 8, 0, kDeviceCoherent);
          __builtin_amdgcn_raw_buffer_store_b32(unit, ws_tag_rsrc, slot * 8 + 4, 0, kDeviceCoherent);
        }
        pub_pending = true;
        pub_unit = unit;
        pub_first = unit_first;
        pub_n = n;
        pub_tiles = gt - seg_g + 1;
      }
      // the next tile starts a new unit: load its Q now, so that it arrives
      // while this workgroup waits for the next tile anyway
      if (gt + 1 < run_e) start_unit(cb, ckvh, cs);
    }

    // ---- the run's last piece is still to be counted
    if (pub_pending) {
      wait_all();
      __syncthreads();
      const int is_last = count_piece();
      if (tid == 0) sh_int[2] = is_last;
      __syncthreads();
      if (sh_int[2]) merge_unit<D>(p, sc, seqs, smem, mark, pub_unit, pub_first, pub_n);
      pub_pending = false;
    }

    // ---- steal: probe tail chunks, the last chunk of every range first.
    // Every workgroup ends on one exhausted probe, also without stealing
    // (nt = 0): the launch's last probe advances the generation, so that no
    // call can mistake a piece tag of an earlier call for one of its own.
    owner = false;
    const int total_probes = sc.Pe * (sc.nt + 1);
    int got = -1;
    for (;;) {
      if (tid == 0) {
        const int k = __hip_atomic_fetch_add(p.thief_ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int res = -2;                                  // chunk taken: probe again
        if (k >= sc.Pe * sc.nt) {
          res = -1;                                    // nothing left
          if (k == total_probes - 1) {                 // the launch's last probe: next call's state
            __hip_atomic_store(p.thief_ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(p.gen, mark, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
        } else {
          const int q = k % sc.Pe;
          const int i = sc.nt - 1 - k / sc.Pe;
          if (claim(q, i)) res = k;
        }
        sh_int[3] = res;
      }
      __syncthreads();
      const int res = sh_int[3];
      __syncthreads();
      if (res != -2) {
        got = res;
        break;
      }
    }
    if (got < 0) break;
    const int q = got % sc.Pe;
    const int i = sc.nt - 1 - got / sc.Pe;
    run_a = sc.sub_begin(q, 1 + i);
    run_e = run_a + sc.cs;
  }
}

// Zero the state region and the piece tags of a workspace.
__global__ void zero_state_kernel(int* state, int n_state, int* tags, int n_tags) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_state) state[i] = 0;
  else if (i - n_state < n_tags) tags[i - n_state] = 0;
}

// ---------------------------------------------------------------- host side

int key_tile(int dtype, int D) {
  const int elt = dtype == SPECMOE_BF16 ? 2 : 4;
  return kTileBytes / (D * elt);
}

// Workspace layout.  The state region has the same layout for every
// descriptor with the same Hkv: generation and probe counter at offset 0,
// claim marks for the largest grid, per-unit counters for the largest launch.
// Only the piece region (tags, lse, O) depends on the grid and the shape, and
// a piece is only read under a tag of the current call's generation.
struct Plan {
  int g, P, Rcap;
  size_t claims_off, counters_off, counter_bytes;   // state region: [0, counter_bytes)
  size_t slots, ws_tag_off, ws_lse_off, ws_o_off, ws_bytes;
};

constexpr int kMaxGrid = 2048;         // merge candidates (10 per range) are flagged in one 34 KB tile buffer

int validate_desc(const specmoe_verify_desc* d) {
  if (!d) return SPECMOE_ERR_NULL_POINTER;
  if (d->dtype != SPECMOE_F32 && d->dtype != SPECMOE_BF16) return SPECMOE_ERR_DTYPE;
  if (d->D != 64 && d->D != 128) return SPECMOE_ERR_HEAD_DIM;
  if (d->B < 0 || d->Hq <= 0 || d->Hkv <= 0 || d->C_max < 1 || d->S_max < d->C_max)
    return SPECMOE_ERR_SHAPE;
  if (d->Hq % d->Hkv != 0) return SPECMOE_ERR_GQA;
  const int64_t g = d->Hq / d->Hkv;
  if ((int64_t)d->C_max * g > kMaxRows) return SPECMOE_ERR_ROWS;
  if (d->flags & ~SPECMOE_DETERMINISTIC) return SPECMOE_ERR_FLAGS;
  if (d->grid_blocks < 0 || d->grid_blocks > kMaxGrid) return SPECMOE_ERR_GRID;
  // partial results are addressed through 32-bit buffer descriptors: up to
  // 10 pieces per workgroup (2 per sub-range, 5 sub-ranges per range)
  const int64_t grid = d->grid_blocks ? d->grid_blocks : kDefaultGrid;
  if (10 * grid * (int64_t)d->C_max * g * d->D * 4 >= ((int64_t)1 << 31)) return SPECMOE_ERR_GRID;
  // index arithmetic: (sequence, token, head) row indices stay in 32 bits,
  // byte offsets inside one (sequence, KV head) slab are 32-bit, packed
  // sequence lengths need T < 2^24, tile counts per launch stay in 32 bits.
  if ((int64_t)d->B * d->C_max * d->Hq >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  const int64_t elt = d->dtype == SPECMOE_BF16 ? 2 : 4;
  if ((int64_t)d->S_max * d->D * elt >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  if (d->S_max >= (1 << 24)) return SPECMOE_ERR_SHAPE;
  const int64_t tile = key_tile(d->dtype, d->D);
  if ((int64_t)kMaxSeqs * d->Hkv * ((d->S_max + tile - 1) / tile) >= ((int64_t)1 << 30)) return SPECMOE_ERR_SHAPE;
  return SPECMOE_OK;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

Plan make_plan(const specmoe_verify_desc* d) {
  Plan pl;
  pl.g = d->Hq / d->Hkv;
  pl.P = d->grid_blocks ? d->grid_blocks : kDefaultGrid;
  pl.Rcap = d->C_max * pl.g;
  pl.claims_off = 256;
  pl.counters_off = pl.claims_off + (size_t)kMaxGrid * 4 * sizeof(int);
  pl.counter_bytes = align256(pl.counters_off + (size_t)kMaxSeqs * d->Hkv * sizeof(int));
  pl.slots = (size_t)10 * pl.P;
  pl.ws_tag_off = pl.counter_bytes;
  pl.ws_lse_off = pl.ws_tag_off + align256(pl.slots * 2 * sizeof(int));
  pl.ws_o_off = pl.ws_lse_off + align256(pl.slots * pl.Rcap * sizeof(float));
  pl.ws_bytes = pl.ws_o_off + pl.slots * pl.Rcap * d->D * sizeof(float);
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
  const int n_state = (int)(pl.counter_bytes / sizeof(int));
  const int n_tags = (int)((pl.ws_lse_off - pl.ws_tag_off) / sizeof(int));
  char* ws = static_cast<char*>(workspace);
  (void)hipGetLastError();
  hipLaunchKernelGGL(zero_state_kernel, dim3((n_state + n_tags + 255) / 256), dim3(256), 0,
                     static_cast<hipStream_t>(stream), reinterpret_cast<int*>(ws), n_state,
                     reinterpret_cast<int*>(ws + pl.ws_tag_off), n_tags);
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
    case SPECMOE_ERR_GRID: return "grid_blocks must be 0 (default) or in [1, 2048], with partial results under 2 GB";
    case SPECMOE_ERR_FLAGS: return "unknown bits in flags";
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
  p.gen = reinterpret_cast<int*>(ws);
  p.thief_ctr = p.gen + 1;
  p.claims = reinterpret_cast<int*>(ws + pl.claims_off);
  p.counters = reinterpret_cast<int*>(ws + pl.counters_off);
  p.ws_tag = reinterpret_cast<int*>(ws + pl.ws_tag_off);
  p.ws_lse = reinterpret_cast<float*>(ws + pl.ws_lse_off);
  p.ws_o = reinterpret_cast<float*>(ws + pl.ws_o_off);
  p.ws_tag_bytes = (int)(pl.ws_lse_off - pl.ws_tag_off);
  p.ws_lse_bytes = (int)(pl.ws_o_off - pl.ws_lse_off);
  p.ws_o_bytes = (int)(pl.ws_bytes - pl.ws_o_off);
  p.deterministic = (desc->flags & SPECMOE_DETERMINISTIC) ? 1 : 0;
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
