// Chunked verification attention for MI355X (gfx950, CDNA4).
//
// Computes, for every sequence b and KV head, softmax(scale*Q K^T + M) V over
// the cached context plus the draft chunk, with a chain mask inside the chunk
// (SpecMoEOff, Section 5.1), and the log-sum-exp of every row.
//
// Design (one GPU stream, two kernels):
//   * Unit of work = (sequence b, KV head).  The c_b draft tokens times the g
//     query heads that share the KV head form the unit's R_b = c_b*g query
//     rows; they are packed into 32-row MFMA tiles, so Q K^T and P V become
//     small dense contractions that reuse every K/V byte for all rows.
//   * Split-KV: the unit's keys [0, T_b) are cut into partitions of `L` keys
//     counted back from T_b, so the chunk's own keys always sit in partition 0
//     and every query row sees at least one key of every partition it is in.
//     One 256-thread workgroup handles one (unit, partition).  Partitioning
//     the sequence needs a combine of partial results, as the paper notes for
//     its sequence-wise KV partition (Section 5.2); it is done with
//     log-sum-exp weights by verify_combine_kernel.
//   * K/V streaming: each workgroup iteration stages a 32 KB K tile and a
//     32 KB V tile in LDS with fully coalesced 16-byte loads (one wave load
//     instruction reads 1 KB of contiguous cache rows); the next tile's loads
//     are in flight in registers while the current tile is consumed.  LDS rows
//     are XOR-swizzled in 16-byte chunks, so the MFMA operand reads are free
//     of bank conflicts.
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

constexpr int kThreads = 256;       // 4 waves of 64
constexpr int kWaves = 4;
constexpr int kSub = 32;            // keys per MFMA subtile
constexpr int kRowTile = 32;        // query rows per MFMA tile
constexpr int kMaxRows = 128;       // row tiles per unit <= 4
constexpr int kTileBytes = 32768;   // K bytes (and V bytes) staged per iteration
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) short i16x8;

struct Params {
  const char* q;
  const char* k;
  const char* v;
  const int32_t* ctx_lens;
  const int32_t* chunk_lens;
  float* out;
  float* lse;
  float* ws_o;      // [units][nsplit][Rcap][D]
  float* ws_lse;    // [units][nsplit][Rcap]
  int B, Hq, Hkv, g, D, C_max, S_max;
  int L;            // keys per split
  int nsplit;       // splits per unit the grid provides
  int Rcap;         // C_max * g
  float sl2;        // scale * log2(e)
};

// Lengths of sequence b, clamped into the documented ranges so that no access
// can leave the buffers even if the caller broke a precondition.
struct Lens {
  int l, c, T;
};

__device__ __forceinline__ Lens load_lens(const Params& p, int b) {
  int c = p.chunk_lens[b];
  int l = p.ctx_lens[b];
  c = c < 0 ? 0 : (c > p.C_max ? p.C_max : c);
  l = l < 0 ? 0 : l;
  if (l > p.S_max - c) l = p.S_max - c;
  Lens r;
  r.l = l;
  r.c = c;
  r.T = l + c;
  return r;
}

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

template <bool BF16, int D>
__global__ __launch_bounds__(kThreads, 2) void verify_main_kernel(Params p) {
  using C = Cfg<BF16, D>;
  __shared__ __attribute__((aligned(16))) char smem[2 * C::kLdsTile];
  char* ks = smem;
  char* vs = smem + C::kLdsTile;

  // split-major 1-D grid: all units' partition 0 first, empty blocks last
  const int units = p.B * p.Hkv;
  const int split = blockIdx.x / units;
  const int unit = blockIdx.x - split * units;
  const int b = unit / p.Hkv;
  const int kvh = unit - b * p.Hkv;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lr = lane & 31;     // row (or key, or d) index inside a 32-wide MFMA block
  const int half = lane >> 5;   // which half of the MFMA k dimension this lane feeds

  const Lens ln = load_lens(p, b);
  const int g = p.g;

  // Padding rows c_b <= i < C_max of this unit's heads: out = 0, lse = -inf.
  if (split == 0) {
    const int pad_rows = (p.C_max - ln.c) * g;
    for (int idx = tid; idx < pad_rows * (D / 4); idx += kThreads) {
      const int row = idx / (D / 4);
      const int d4 = idx - row * (D / 4);
      const int i = ln.c + row / g;
      const int h = kvh * g + row % g;
      float* o = p.out + ((size_t)(b * p.C_max + i) * p.Hq + h) * D + 4 * d4;
      *reinterpret_cast<f32x4*>(o) = f32x4{0.f, 0.f, 0.f, 0.f};
      if (d4 == 0) p.lse[(size_t)(b * p.C_max + i) * p.Hq + h] = -INFINITY;
    }
  }
  if (ln.c == 0) return;
  const int nsplit_b = (ln.T + p.L - 1) / p.L;
  if (split >= nsplit_b) return;

  const int hi = ln.T - split * p.L;
  const int lo = hi > p.L ? hi - p.L : 0;
  const int R = ln.c * g;
  const int n_rt = (R + kRowTile - 1) / kRowTile;
  const int n_rt4 = n_rt == 3 ? 4 : n_rt;
  const int n_kg = kWaves / n_rt4;
  const int rt = wave % n_rt4;
  const int kg = wave / n_rt4;
  const bool has_rows = rt < n_rt;

  // ---- Q operand: lane holds row rt*32+lr, chunks 2j+half of its D values.
  const int row = rt * kRowTile + lr;
  const bool row_valid = has_rows && row < R;
  const int tok = row_valid ? row / g : 0;
  const int vis = row_valid ? ln.l + tok : 0x7fffffff;   // last visible key
  u32x4 qreg[C::kQChunks];
  {
    const char* qrow = p.q + ((size_t)(b * p.C_max + tok) * p.Hq + kvh * g + (row_valid ? row % g : 0)) *
                                 C::kRowBytes;
#pragma unroll
    for (int j = 0; j < C::kQChunks; ++j) {
      qreg[j] = row_valid ? *reinterpret_cast<const u32x4*>(qrow + 16 * (2 * j + half))
                          : u32x4{0u, 0u, 0u, 0u};
    }
  }

  f32x16 o[C::kDC];
#pragma unroll
  for (int dc = 0; dc < C::kDC; ++dc) o[dc] = f32x16{};
  float m_run = -INFINITY;   // running row max, in log2 units
  float l_run = 0.f;         // running row sum of 2^(s - m_run)

  // The unit's K and V slabs; offsets inside a slab fit in 32 bits (checked
  // on the host), so the loads use a uniform base plus a 32-bit offset.
  const size_t kv_base = ((size_t)b * p.Hkv + kvh) * (size_t)p.S_max * C::kRowBytes;
  const char* __restrict__ kg_ptr = p.k + kv_base;
  const char* __restrict__ vg_ptr = p.v + kv_base;

  // Prefetch registers.  Load j of thread tid takes row j*kRowsPerPass + r0,
  // chunk c0: one wave instruction reads 1 KB of contiguous cache rows.
  const int r0 = tid / C::kChunks;
  const int c0 = tid % C::kChunks;
  u32x4 kreg[C::kLoads], vreg[C::kLoads];
  auto prefetch = [&](int k0, int nk) {
    const uint32_t base = (uint32_t)(k0 + r0) * C::kRowBytes + 16u * c0;
#pragma unroll
    for (int j = 0; j < C::kLoads; ++j) {
      const uint32_t off = base + (uint32_t)(j * C::kRowsPerPass * C::kRowBytes);
      if (j * C::kRowsPerPass + r0 < nk) {
        kreg[j] = *reinterpret_cast<const u32x4*>(kg_ptr + off);
        vreg[j] = *reinterpret_cast<const u32x4*>(vg_ptr + off);
      } else {
        kreg[j] = u32x4{0u, 0u, 0u, 0u};
        vreg[j] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto stage = [&]() {
    const int base = lds_off<C>(r0, c0);
#pragma unroll
    for (int j = 0; j < C::kLoads; ++j) {
      const int off = base + j * C::kRowsPerPass * C::kPitch;
      *reinterpret_cast<u32x4*>(ks + off) = kreg[j];
      *reinterpret_cast<u32x4*>(vs + off) = vreg[j];
    }
  };

  const int ntiles = (hi - lo + C::kTileKeys - 1) / C::kTileKeys;
  prefetch(lo, hi - lo < C::kTileKeys ? hi - lo : C::kTileKeys);

  for (int t = 0; t < ntiles; ++t) {
    const int k0 = lo + t * C::kTileKeys;
    const int nk = hi - k0 < C::kTileKeys ? hi - k0 : C::kTileKeys;
    __syncthreads();   // every wave is done reading the previous tile
    stage();
    __syncthreads();
    if (t + 1 < ntiles) {
      const int k1 = k0 + C::kTileKeys;
      prefetch(k1, hi - k1 < C::kTileKeys ? hi - k1 : C::kTileKeys);
    }
    if (!has_rows) continue;

    for (int sub = kg; sub < C::kNSub; sub += n_kg) {
      if (sub * kSub >= nk) break;
      const int key0 = k0 + sub * kSub;            // absolute index of the subtile's key 0
      const int krow = sub * kSub + lr;            // this lane's K row in the tile

      // ---- S^T = K Q^T for 32 keys x 32 rows.
      f32x16 s = f32x16{};
#pragma unroll
      for (int j = 0; j < C::kQChunks; ++j) {
        const u32x4 kop = *reinterpret_cast<const u32x4*>(ks + lds_off<C>(krow, 2 * j + half));
        if constexpr (BF16) {
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kop),
                                                      __builtin_bit_cast(bf16x8, qreg[j]), s, 0, 0, 0);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            s = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(kop[e]), __uint_as_float(qreg[j][e]),
                                                     s, 0, 0, 0);
        }
      }

      // ---- scale, mask, online softmax.  Lane holds row `row`, keys
      // key0 + 8*(r/4) + 4*half + r%4 for r = 0..15.
      const bool edge = (key0 + kSub > hi) || (key0 + kSub - 1 > ln.l);
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = s[r] * p.sl2;
        if (edge) {
          const int key = key0 + 8 * (r >> 2) + 4 * half + (r & 3);
          if (key >= hi || key > vis) x = -INFINITY;
        }
        s[r] = x;
        mx = fmaxf(mx, x);
      }
      mx = fmaxf(mx, xor32(mx));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      float rs = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = __builtin_amdgcn_exp2f(s[r] - m_use);
        rs += s[r];
      }
      rs += xor32(rs);
      l_run = l_run * alpha + rs;
      m_run = m_new;
#pragma unroll
      for (int dc = 0; dc < C::kDC; ++dc) o[dc] *= alpha;

      // ---- O^T += V^T P^T.
      if constexpr (BF16) {
        u32x4 pb[2];
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
          for (int w = 0; w < 4; ++w) pb[t2][w] = pack_bf16x2(s[8 * t2 + 2 * w], s[8 * t2 + 2 * w + 1]);
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
            o[dc] = __builtin_amdgcn_mfma_f32_32x32x2f32(x, s[u], o[dc], 0, 0, 0);
          }
        }
      }
    }
  }

  // ---- merge the key groups of each row tile through LDS.
  if (n_kg > 1) {
    __syncthreads();
    float* mbuf = reinterpret_cast<float*>(smem);
    // region of wave (kg, rt), kg >= 1: stats (2 x 64 floats) then O (kDC*16*64)
    constexpr int kRegion = 128 + C::kDC * 16 * 64;
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
  if (kg != 0 || !row_valid) return;

  // ---- write: normalised rows and natural-log lse.  Every valid row saw at
  // least one key of this partition, so l_run > 0.
  const float inv = 1.f / l_run;
  const float lse_val = (m_run + log2f(l_run)) * kLn2;
  float* dst;
  size_t lse_idx;
  const int hq = kvh * g + row % g;
  if (nsplit_b == 1) {
    dst = p.out + ((size_t)(b * p.C_max + tok) * p.Hq + hq) * D;
    lse_idx = (size_t)(b * p.C_max + tok) * p.Hq + hq;
    if (half == 0) p.lse[lse_idx] = lse_val;
  } else {
    const size_t slot = ((size_t)unit * p.nsplit + split) * p.Rcap + row;
    dst = p.ws_o + slot * D;
    if (half == 0) p.ws_lse[slot] = lse_val;
  }
#pragma unroll
  for (int dc = 0; dc < C::kDC; ++dc)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d0 = dc * 32 + 8 * g4 + 4 * half;
      f32x4 val = {o[dc][4 * g4] * inv, o[dc][4 * g4 + 1] * inv, o[dc][4 * g4 + 2] * inv,
                   o[dc][4 * g4 + 3] * inv};
      *reinterpret_cast<f32x4*>(dst + d0) = val;
    }
}

// Combine the per-partition results of units that have more than one
// partition: lse = log sum_s exp(lse_s), out = sum_s exp(lse_s - lse) * O_s.
template <int D>
__global__ __launch_bounds__(kThreads) void verify_combine_kernel(Params p) {
  constexpr int kTPR = D / 4;                  // threads per row (float4 each)
  constexpr int kRowsPerPass = kThreads / kTPR;
  const int unit = blockIdx.x;
  const int b = unit / p.Hkv;
  const int kvh = unit - b * p.Hkv;
  const Lens ln = load_lens(p, b);
  if (ln.c == 0) return;
  const int ns = (ln.T + p.L - 1) / p.L;
  if (ns <= 1) return;
  const int R = ln.c * p.g;
  const int d0 = 4 * (threadIdx.x % kTPR);
  for (int row = threadIdx.x / kTPR; row < R; row += kRowsPerPass) {
    const size_t base = (size_t)unit * p.nsplit * p.Rcap + row;
    float M = -INFINITY;
    for (int s = 0; s < ns; ++s) M = fmaxf(M, p.ws_lse[base + (size_t)s * p.Rcap]);
    float Z = 0.f;
    for (int s = 0; s < ns; ++s) Z += expf(p.ws_lse[base + (size_t)s * p.Rcap] - M);
    const float lse_val = M + logf(Z);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < ns; ++s) {
      const size_t slot = base + (size_t)s * p.Rcap;
      const float w = expf(p.ws_lse[slot] - lse_val);
      const f32x4 x = *reinterpret_cast<const f32x4*>(p.ws_o + slot * D + d0);
      acc += w * x;
    }
    const int tok = row / p.g;
    const int hq = kvh * p.g + row % p.g;
    const size_t orow = (size_t)(b * p.C_max + tok) * p.Hq + hq;
    *reinterpret_cast<f32x4*>(p.out + orow * D + d0) = acc;
    if (d0 == 0) p.lse[orow] = lse_val;
  }
}

// ---------------------------------------------------------------- host side

int key_tile(int dtype, int D) {
  const int elt = dtype == SPECMOE_BF16 ? 2 : 4;
  return kTileBytes / (D * elt);
}

struct Plan {
  int g, L, nsplit, Rcap;
  size_t ws_o_bytes, ws_lse_off, ws_bytes;
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
  // index arithmetic: products of (b, token, head) counts stay in 32 bits,
  // byte offsets are 64-bit.
  if ((int64_t)d->B * d->C_max * d->Hq >= (int64_t)1 << 31) return SPECMOE_ERR_SHAPE;
  if ((int64_t)d->B * d->Hkv >= (int64_t)1 << 31) return SPECMOE_ERR_SHAPE;
  // byte offsets inside one (sequence, KV head) slab are 32-bit in the kernel
  const int64_t elt = d->dtype == SPECMOE_BF16 ? 2 : 4;
  if ((int64_t)d->S_max * d->D * elt >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;
  const int tile = key_tile(d->dtype, d->D);
  if (d->split_len != 0 && (d->split_len < 0 || d->split_len % tile != 0 || d->split_len < d->C_max))
    return SPECMOE_ERR_SPLIT;
  return SPECMOE_OK;
}

// Split length: aim at ~2048 workgroups for caches that are full up to S_max,
// in whole key tiles, at least one tile, at least C_max keys.
int choose_split(const specmoe_verify_desc* d) {
  if (d->split_len != 0) return d->split_len;
  const int tile = key_tile(d->dtype, d->D);
  const int64_t units = (int64_t)d->B * d->Hkv;
  int64_t L = ((int64_t)d->S_max * units + 2047) / 2048;
  L = (L + tile - 1) / tile * tile;
  const int64_t lmin = ((int64_t)d->C_max + tile - 1) / tile * tile;
  const int64_t lmax = ((int64_t)d->S_max + tile - 1) / tile * tile;
  if (L < lmin) L = lmin;
  if (L > lmax) L = lmax;
  if (L < lmin) L = lmin;
  return (int)L;
}

Plan make_plan(const specmoe_verify_desc* d) {
  Plan pl;
  pl.g = d->Hq / d->Hkv;
  pl.L = choose_split(d);
  pl.nsplit = (d->S_max + pl.L - 1) / pl.L;
  pl.Rcap = d->C_max * pl.g;
  const size_t units = (size_t)d->B * d->Hkv;
  if (pl.nsplit <= 1 || units == 0) {
    pl.ws_o_bytes = pl.ws_lse_off = pl.ws_bytes = 0;
    return pl;
  }
  const size_t slots = units * pl.nsplit * pl.Rcap;
  pl.ws_o_bytes = slots * d->D * sizeof(float);
  pl.ws_lse_off = (pl.ws_o_bytes + 255) / 256 * 256;
  pl.ws_bytes = pl.ws_lse_off + slots * sizeof(float);
  return pl;
}

template <bool BF16, int D>
void launch(const Params& p, const Plan& pl, hipStream_t stream, const specmoe_verify_desc* d) {
  const dim3 grid(pl.nsplit * p.B * p.Hkv);
  if (d->ev_main_begin) (void)hipEventRecord(static_cast<hipEvent_t>(d->ev_main_begin), stream);
  hipLaunchKernelGGL((verify_main_kernel<BF16, D>), grid, dim3(kThreads), 0, stream, p);
  if (d->ev_main_end) (void)hipEventRecord(static_cast<hipEvent_t>(d->ev_main_end), stream);
  if (pl.nsplit > 1)
    hipLaunchKernelGGL((verify_combine_kernel<D>), dim3(p.B * p.Hkv), dim3(kThreads), 0, stream, p);
}

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

}  // namespace

extern "C" {

size_t specmoe_verify_attn_workspace_bytes(const specmoe_verify_desc* desc) {
  if (validate_desc(desc) != SPECMOE_OK) return 0;
  return make_plan(desc).ws_bytes;
}

int32_t specmoe_verify_attn_split_len(const specmoe_verify_desc* desc) {
  const int st = validate_desc(desc);
  if (st != SPECMOE_OK) return st;
  return choose_split(desc);
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
    case SPECMOE_ERR_SPLIT: return "split_len must be 0 or a multiple of the key tile that is >= C_max";
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
  int st = validate_desc(desc);
  if (st != SPECMOE_OK) return st;
  if (desc->B == 0) return SPECMOE_OK;   // nothing to read or write
  if (!q || !k_cache || !v_cache || !ctx_lens || !chunk_lens || !out || !lse) return SPECMOE_ERR_NULL_POINTER;
  if (!isfinite(scale)) return SPECMOE_ERR_SCALE;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out)) return SPECMOE_ERR_ALIGN;
  const Plan pl = make_plan(desc);
  if (pl.ws_bytes > 0) {
    if (!desc->workspace) return SPECMOE_ERR_NULL_POINTER;
    if (!aligned16(desc->workspace)) return SPECMOE_ERR_ALIGN;
    if (desc->workspace_bytes < pl.ws_bytes) return SPECMOE_ERR_WORKSPACE;
  }
  if ((int64_t)pl.nsplit * desc->B * desc->Hkv >= ((int64_t)1 << 31)) return SPECMOE_ERR_SHAPE;

  Params p;
  p.q = static_cast<const char*>(q);
  p.k = static_cast<const char*>(k_cache);
  p.v = static_cast<const char*>(v_cache);
  p.ctx_lens = ctx_lens;
  p.chunk_lens = chunk_lens;
  p.out = out;
  p.lse = lse;
  p.ws_o = pl.ws_bytes ? static_cast<float*>(desc->workspace) : nullptr;
  p.ws_lse = pl.ws_bytes ? reinterpret_cast<float*>(static_cast<char*>(desc->workspace) + pl.ws_lse_off) : nullptr;
  p.B = desc->B;
  p.Hq = desc->Hq;
  p.Hkv = desc->Hkv;
  p.g = pl.g;
  p.D = desc->D;
  p.C_max = desc->C_max;
  p.S_max = desc->S_max;
  p.L = pl.L;
  p.nsplit = pl.nsplit;
  p.Rcap = pl.Rcap;
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
