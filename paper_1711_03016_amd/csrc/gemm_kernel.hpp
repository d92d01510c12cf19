// Dense-layer matrix products on gfx950 matrix cores, with fused epilogues.
//
// The one kernel template computes C[M,N] = sum_k A(m,k) B(k,n) for the three
// operand layouts a dense layer and its adjoint need (the adjoint of dot,
// dA = dC.B^T and dB = A^T.dC, never materialises a transpose):
//   NN  forward               A = X [M,K] (k contiguous), B = W [K,N] (n contiguous)
//   NT  adjoint wrt input     A = dY [M,N'] (k contiguous), B = W [K',N'] read as W^T (k contiguous)
//   TN  adjoint wrt weights   A = X [K,M] read as X^T (m contiguous), B = dY [K,N] (n contiguous)
// and fuses the element-wise work around the product into the same kernel
// (linear-algebra and element-wise fusion, DLVM sections 1 and 3.1.2):
//   NN  H = act(alpha * acc + bias[n])                         (bias + activation)
//   NT  dX = acc * act'(Hprev) + R, act' from the saved output (adjoint of act;
//       R is another adjoint contribution to the same value, accumulated)
//   TN  dW = acc (float32); db[n] = sum_k B(k,n) by the first row of tiles
//       (the padded ones-row of [X 1]^T.dY, without materialising it)
//
// Data movement. Every operand tile is staged in LDS as rows of 128 bytes of
// the reduction dimension (32 float32 or 64 bf16), one row per m (or n)
// index, padded to a 144-byte stride. Global loads are 16 bytes per lane when
// the operand's contiguous extent allows it (per operand), else element by
// element with bounds checks. An operand whose reduction dimension is strided
// in memory (the TN layout, and W in the NN layout) is transposed in registers
// on its way to LDS (4x4 float32 blocks are a register renaming; 8x8 bf16
// blocks use byte permutes), so the MFMA fragment of every lane is one
// 16-byte LDS read in all layouts. The lane-to-chunk assignment (chunk index
// fastest) together with the 144-byte stride keeps both those stores and the
// fragment reads free of LDS bank conflicts. The next k-tile is prefetched into
// registers while the current one is multiplied from LDS; LDS is
// double-buffered so one barrier per k-tile suffices.
//
// Matrix cores: float32 uses v_mfma_f32_32x32x2_f32 (one 16-byte fragment =
// 4 consecutive k per lane feeds 4 instructions), bf16 uses
// v_mfma_f32_32x32x16_bf16 (8 consecutive k per lane feed one instruction).
// Inside one fragment the assignment of k values to instruction slots is a
// permutation applied identically to both operands, which leaves the sum
// unchanged.
//
// Splitting the reduction inside a workgroup. For small products a workgroup
// of WK groups of waves covers one output tile: every group multiplies the
// same LDS tiles but takes every WK-th k-step of them, and at the end the
// groups' accumulators are added through LDS in increasing group order before
// the epilogue. This keeps all four SIMDs of a compute unit busy on a small
// tile without any cross-workgroup communication, and the sum order is fixed.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace dlvm {
namespace gemm {

constexpr int kRowStride = 144;  // bytes per LDS row: 128 bytes of k plus 16 of padding
constexpr int kChunks = 8;       // 16-byte chunks of k per LDS row

enum Epi { EPI_STORE = 0, EPI_DACT = 1, EPI_DW = 2, EPI_CHAIN = 3 };

template <typename T> struct Elem;
template <> struct Elem<float> { static constexpr int VW = 4; static constexpr int BK = 32; };
template <> struct Elem<bf16_t> { static constexpr int VW = 8; static constexpr int BK = 64; };

struct Params {
  int64_t M, N, K;
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  void* C; int64_t ldc;
  const void* bias;
  const void* aux;
  const void* residual;
  float* colsum;
  float alpha;
  int act;
  int tiles_m, tiles_n;
  int64_t nvec;  // entries of bias / colsum (columns n >= nvec have none)
  uint32_t a_bytes, b_bytes;  // extents of A and B in bytes (buffer-descriptor kernels)
  uint32_t a2_bytes;          // extent of A2 (k-slices of a two-phase product), or 0
  // Split reduction (adjoint wrt the weights): workgroup b handles tile
  // b % (tiles_m * tiles_n) over k-slice b / (tiles_m * tiles_n) of k_chunk
  // k, and writes its float32 partial product (and partial column sums) at
  // C + slice * c_split (colsum + slice * cs_split). splits == 1: no split.
  int splits;
  int64_t k_chunk, c_split, cs_split;
  // Two-phase contraction (a sum of two products accumulated in one pass,
  // sum_k over [A A2] . B): k < K1 reads A (row stride lda) at k, k >= K1
  // reads A2 (row stride lda2) at k - K1; B runs through all K. K1 == K (and
  // A2 null): one phase.
  const void* A2;
  int64_t lda2, K1;
  int res_pre;  // EPI_DACT: (acc + R) * act'(Hprev) instead of acc * act'(Hprev) + R
  // EPI_CHAIN (float32 NN): the eight-operator chain on z = acc with bias[n]
  // and x_skip = aux (same shape as C): C receives zbar, C2 xbar, and each
  // wavefront of tile t writes its sum of e^2 to partials[t * WM * WN + wave].
  void* C2;
  float* partials;
  float inv_n;
  // Rectifier masks in accumulator order (direct-to-LDS kernel, 256 x 256
  // tiles on 2 x 4 waves or 64 x 128 tiles on 2 x 2 waves, unsplit; null:
  // none). With W = TM * TN / 2 words per lane (4 and 1) and T threads, tile
  // (tm, tn) owns T x W words from (tm * tiles_n + tn) * T * W; lane t of the
  // workgroup owns words W t .. W t + W - 1, whose bit 16 q + r (in word q / 2
  // for q odd, shifted) is element r of the lane's accumulator block
  // q = i * TN + j. EPI_STORE with the rectifier writes bit = (stored output
  // > 0); EPI_DACT reads it in place of the saved activation.
  uint32_t* mask;
};

// Source of pipeline stage kt (KSTAGE k per stage) of a two-phase
// contraction: the stages of phase 1 cover [0, K1) and those of phase 2
// [K1, K), each phase starting on a stage boundary (its last stage is padded
// with zeros by the loader).
template <typename T, bool BKM>
struct StageSrc {
  const T* a;
  int64_t lda;
  const T* b;
  int64_t k0, klim;
};
// PH2 false: the product has one phase (A2 unused) and no per-stage choice is made.
template <typename T, bool BKM, bool PH2>
__device__ __forceinline__ StageSrc<T, BKM> stage_src(const Params& p, const T* A, const T* B,
                                                      int64_t kt, int64_t nk1, int64_t kstage) {
  StageSrc<T, BKM> s;
  if constexpr (!PH2) {
    s.a = A; s.lda = p.lda; s.b = B; s.k0 = kt * kstage; s.klim = p.K;
    return s;
  }
  const bool ph2 = kt >= nk1;
  s.a = ph2 ? static_cast<const T*>(p.A2) : A;
  s.lda = ph2 ? p.lda2 : p.lda;
  s.b = ph2 ? B + (BKM ? p.K1 : p.K1 * p.ldb) : B;
  s.k0 = (ph2 ? kt - nk1 : kt) * kstage;
  s.klim = ph2 ? p.K - p.K1 : p.K1;
  return s;
}

// Tile index of workgroup `bid` of a product; with a split reduction, also
// narrows p to the workgroup's k-slice and partial outputs.
template <typename T, bool AK, bool BKM>
__device__ __forceinline__ int split_slice(Params& p, int bid) {
  if (p.splits > 1) {
    const int tiles = p.tiles_m * p.tiles_n;
    const int sl = bid / tiles;
    bid -= sl * tiles;
    const int64_t k0 = static_cast<int64_t>(sl) * p.k_chunk;
    const int64_t kl = p.K - k0 < p.k_chunk ? p.K - k0 : p.k_chunk;
    int64_t sa = AK ? k0 : k0 * p.lda;
    const int64_t sb = BKM ? k0 : k0 * p.ldb;
    if (p.A2 != nullptr && k0 >= p.K1) {
      // a slice of the second phase (slices never straddle K1)
      p.A = p.A2;
      p.lda = p.lda2;
      sa = AK ? k0 - p.K1 : (k0 - p.K1) * p.lda2;
      if (p.a_bytes != 0u) p.a_bytes = p.a2_bytes;
    }
    p.A = static_cast<const T*>(p.A) + sa;
    p.B = static_cast<const T*>(p.B) + sb;
    // (extents of the buffer-descriptor loads; 0 means none and stays 0)
    if (p.a_bytes != 0u) p.a_bytes -= static_cast<uint32_t>(sa * static_cast<int64_t>(sizeof(T)));
    if (p.b_bytes != 0u) p.b_bytes -= static_cast<uint32_t>(sb * static_cast<int64_t>(sizeof(T)));
    p.K = kl;
    p.K1 = kl;  // split products have one phase
    p.C = static_cast<float*>(p.C) + sl * p.c_split;
    if (p.colsum != nullptr) p.colsum += sl * p.cs_split;
  }
  return bid;
}

// Tile order. Workgroups are dealt round-robin over the 8 XCDs, each with its
// own L2; the tile index is remapped so that each XCD gets a contiguous range
// of tiles, and within a range tiles are visited in bands of 8 tile-rows, so
// the workgroups of one XCD share A and B tiles in its L2 (and each XCD reads
// only part of each operand).
constexpr int kXcds = 8;

// Tile (tm, tn) of workgroup `bid`.
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nt = tiles_m * tiles_n;
  int t = bid;
  if (nt % kXcds == 0) t = (bid % kXcds) * (nt / kXcds) + bid / kXcds;
  constexpr int GM = 8;
  const int band = t / (GM * tiles_n);
  const int first = band * GM;
  const int rows = tiles_m - first < GM ? tiles_m - first : GM;
  const int r = t - band * GM * tiles_n;
  tm = first + r % rows;
  tn = r / rows;
}

__device__ __forceinline__ uint32_t perm_b32(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// One operand tile of ROWS x (KSEG * BK): element (r, k) of the operand is
//   KMAJ:  P[r * ld + k]   (k contiguous)
//   !KMAJ: P[k * ld + r]   (r contiguous)
// and lands in LDS segment (k / BK) % KSEG, row r, byte (k % BK) * sizeof(T).
//
// load() only issues the global loads of the next stage; store() (after the
// current stage has been multiplied) zeroes out-of-range chunks, transposes
// r-contiguous blocks and writes LDS. With 16-byte loads every load is issued
// unconditionally from a clamped, always valid address and its validity is
// kept aside, so no branch and no consumer of the loaded registers sits
// between the loads and the matrix-core work that hides their latency.
template <typename T, bool KMAJ, int ROWS, int THREADS, bool VEC, int KSEG>
struct TileLoader {
  static constexpr int VW = Elem<T>::VW;
  static constexpr int CH = kChunks * KSEG;  // 16-byte chunks of k per row and stage
  static constexpr int TASKS = KMAJ ? ROWS * CH : (ROWS / VW) * CH;
  static constexpr int PER_THREAD = (TASKS + THREADS - 1) / THREADS;
  static constexpr int NLOAD = KMAJ ? PER_THREAD : PER_THREAD * VW;  // 16-byte loads per thread
  static_assert(NLOAD <= 32, "validity mask");
  uint32_t raw[NLOAD][4];
  uint32_t ok = 0;  // bit i: load i lies inside the operand

  // Task q -> (row or row block, chunk). K-contiguous operands put the chunk
  // index fastest (consecutive lanes read consecutive 16 bytes of a row);
  // r-contiguous operands put the 8 chunks of a segment fastest, then the row
  // blocks, then the segment (each k row is read in 128-byte runs).
  __device__ __forceinline__ static void task(int q, int& rowblk, int& c) {
    if constexpr (KMAJ) {
      rowblk = q / CH;
      c = q % CH;
    } else {
      constexpr int RB = ROWS / VW;
      const int c8 = q % kChunks;
      rowblk = (q / kChunks) % RB;
      c = (q / (kChunks * RB)) * kChunks + c8;
    }
  }

  __device__ __forceinline__ void put(int i, const uint4& x) {
    raw[i][0] = x.x; raw[i][1] = x.y; raw[i][2] = x.z; raw[i][3] = x.w;
  }

  __device__ __forceinline__ void load(const T* __restrict__ P, int64_t ld, int64_t r0,
                                       int64_t rlim, int64_t k0, int64_t klim, int tid) {
    ok = 0;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int q = tid + i * THREADS;
      if (TASKS % THREADS != 0 && q >= TASKS) break;
      int rb, c;
      task(q, rb, c);
      if constexpr (KMAJ) {
        const int64_t gr = r0 + rb;
        const int64_t gk = k0 + c * VW;
        if constexpr (VEC) {
          const bool in = gr < rlim && gk < klim;
          ok |= in ? (1u << i) : 0u;
          put(i, *reinterpret_cast<const uint4*>(in ? P + gr * ld + gk : P));
        } else {
          T e[VW];
#pragma unroll
          for (int j = 0; j < VW; ++j)
            e[j] = (gr < rlim && gk + j < klim) ? P[gr * ld + gk + j] : T(0);
          const uint32_t* w = reinterpret_cast<const uint32_t*>(e);
          raw[i][0] = w[0]; raw[i][1] = w[1]; raw[i][2] = w[2]; raw[i][3] = w[3];
          ok |= 1u << i;
        }
      } else {
        const int64_t gr = r0 + rb * VW;
        const int64_t gk = k0 + c * VW;
#pragma unroll
        for (int kk = 0; kk < VW; ++kk) {
          if constexpr (VEC) {
            // The whole 16-byte run lies inside row gk+kk (ld is a multiple of
            // the vector width); elements past rlim reach only outputs that
            // are not stored.
            const bool in = gr < rlim && gk + kk < klim;
            ok |= in ? (1u << (i * VW + kk)) : 0u;
            put(i * VW + kk, *reinterpret_cast<const uint4*>(in ? P + (gk + kk) * ld + gr : P));
          } else {
            T e[VW];
#pragma unroll
            for (int j = 0; j < VW; ++j)
              e[j] = (gr + j < rlim && gk + kk < klim) ? P[(gk + kk) * ld + gr + j] : T(0);
            const uint32_t* w = reinterpret_cast<const uint32_t*>(e);
            const int n = i * VW + kk;
            raw[n][0] = w[0]; raw[n][1] = w[1]; raw[n][2] = w[2]; raw[n][3] = w[3];
            ok |= 1u << n;
          }
        }
      }
    }
  }

  // `lds` is this operand's row 0 in segment 0; segments are SEG_BYTES apart.
  template <int SEG_BYTES>
  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int q = tid + i * THREADS;
      if (TASKS % THREADS != 0 && q >= TASKS) break;
      int rb, c;
      task(q, rb, c);
      char* base = lds + (c / kChunks) * SEG_BYTES + (c % kChunks) * 16;
      if constexpr (KMAJ) {
        const bool o = (ok >> i) & 1u;
        *reinterpret_cast<uint4*>(base + rb * kRowStride) =
            make_uint4(o ? raw[i][0] : 0u, o ? raw[i][1] : 0u, o ? raw[i][2] : 0u,
                       o ? raw[i][3] : 0u);
      } else {
        uint32_t w[VW][4];  // w[kk] = elements (k = kk, r = 0 .. VW-1) of the block
#pragma unroll
        for (int kk = 0; kk < VW; ++kk) {
          const int n = i * VW + kk;
          const bool o = (ok >> n) & 1u;
          w[kk][0] = o ? raw[n][0] : 0u; w[kk][1] = o ? raw[n][1] : 0u;
          w[kk][2] = o ? raw[n][2] : 0u; w[kk][3] = o ? raw[n][3] : 0u;
        }
        uint32_t t[VW][4];  // t[j] = row r = j of the block, its VW k values
        if constexpr (sizeof(T) == 4) {
          // 4x4 float32 transpose: a register renaming.
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) t[j][kk] = w[kk][j];
        } else {
          // 8x8 bf16 transpose: row j, dword p = (k = 2p, k = 2p+1), by byte permutes.
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int p = 0; p < 4; ++p)
              t[j][p] = perm_b32(w[2 * p + 1][j >> 1], w[2 * p][j >> 1],
                                 (j & 1) ? 0x07060302u : 0x05040100u);
        }
#pragma unroll
        for (int j = 0; j < VW; ++j)
          *reinterpret_cast<uint4*>(base + (rb * VW + j) * kRowStride) =
              make_uint4(t[j][0], t[j][1], t[j][2], t[j][3]);
      }
    }
  }
};

template <typename T>
__device__ __forceinline__ void mfma_frag(f32x16& acc, const uint4& a, const uint4& b);

template <>
__device__ __forceinline__ void mfma_frag<float>(f32x16& acc, const uint4& a, const uint4& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ void mfma_frag<bf16_t>(f32x16& acc, const uint4& a, const uint4& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

// Epilogue of one 32 x 32 accumulator block whose first output is (r0, c0).
// Accumulator register r of the block holds row 8*(r/4) + 4*(lane/32) + r%4
// and column lane%32. A block that lies entirely inside the output takes an
// unguarded path; the saved activation and residual of 8 registers are loaded
// before their results are stored, so those loads are in flight together.
template <typename T, typename TO, int EPI>
__device__ __forceinline__ void store_block(const Params& p, const f32x16& acc, int64_t r0,
                                            int64_t c0, int lane) {
  const int64_t col = c0 + (lane & 31);
  const int64_t rb = r0 + 4 * (lane >> 5);
  const bool full = r0 + 32 <= p.M && c0 + 32 <= p.N;
  const bool col_ok = col < p.N;
  const int ld = static_cast<int>(p.ldc);
  float bias_v = 0.0f;
  if constexpr (EPI == EPI_STORE) {
    if (p.bias != nullptr && col < p.nvec) bias_v = load_as_f32<T>(static_cast<const T*>(p.bias) + col);
  }
  const int64_t base = rb * p.ldc + col;  // element (rb, col); rows past M are never dereferenced
  TO* __restrict__ C = static_cast<TO*>(p.C) + base;
  const T* __restrict__ aux = static_cast<const T*>(p.aux);
  const TO* __restrict__ res = static_cast<const TO*>(p.residual);
  const bool has_act = p.act != ACT_NONE;
  if (full) {
#pragma unroll
    for (int h = 0; h < 16; h += 8) {
      float g[8], rv[8];
      if constexpr (EPI == EPI_DACT) {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          const int ro = 8 * ((h + r) >> 2) + (r & 3);
          g[r] = has_act ? load_as_f32<T>(aux + base + ro * ld) : 0.0f;
          rv[r] = res != nullptr ? load_as_f32<TO>(res + base + ro * ld) : 0.0f;
        }
      }
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int ro = 8 * ((h + r) >> 2) + (r & 3);
        float v = acc[h + r];
        if constexpr (EPI == EPI_STORE) {
          v = apply_act(p.act, p.alpha * v + bias_v);
        } else if constexpr (EPI == EPI_DACT) {
          if (p.res_pre) v += rv[r];
          if (has_act) v *= act_grad_from_output(p.act, g[r]);
          if (!p.res_pre) v += rv[r];
        }
        C[ro * ld] = store_cast<TO>(v);
      }
    }
  } else if (col_ok) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int ro = 8 * (r >> 2) + (r & 3);
      if (rb + ro >= p.M) continue;
      float v = acc[r];
      if constexpr (EPI == EPI_STORE) {
        v = apply_act(p.act, p.alpha * v + bias_v);
      } else if constexpr (EPI == EPI_DACT) {
        const float rr = res != nullptr ? load_as_f32<TO>(res + base + ro * ld) : 0.0f;
        if (p.res_pre) v += rr;
        if (has_act) v *= act_grad_from_output(p.act, load_as_f32<T>(aux + base + ro * ld));
        if (!p.res_pre) v += rr;
      }
      C[ro * ld] = store_cast<TO>(v);
    }
  }
}

// The chain epilogue of one 32 x 32 accumulator block (EPI_CHAIN): per
// element the standalone chain kernel's arithmetic (chain_elem), outputs
// zbar and xbar; returns this lane's sum of e^2 over the block.
__device__ __forceinline__ float chain_block(const Params& p, const f32x16& acc, int64_t r0,
                                             int64_t c0, int lane) {
  const int64_t col = c0 + (lane & 31);
  const int64_t rb = r0 + 4 * (lane >> 5);
  if (col >= p.N) return 0.0f;
  const float b = static_cast<const float*>(p.bias)[col];
  const float* __restrict__ xs = static_cast<const float*>(p.aux);
  float* __restrict__ zb = static_cast<float*>(p.C);
  float* __restrict__ xb = static_cast<float*>(p.C2);
  float sq = 0.0f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int64_t row = rb + 8 * (r >> 2) + (r & 3);
    if (row >= p.M) continue;
    const int64_t i = row * p.ldc + col;
    float zo, xo, eo;
    sq += chain_elem(acc[r], b, xs[i], p.inv_n, false, zo, xo, eo);
    zb[i] = zo;
    xb[i] = xo;
  }
  return sq;
}

// LDS bytes of one workgroup of the register-staged kernel.
template <typename T, int BM, int BN, int WK, int KSEG>
constexpr int gemm_smem_bytes() {
  constexpr int stage = KSEG * (BM + BN) * kRowStride;
  constexpr int red = (WK - 1) * BM * BN * 4;
  return 2 * stage > red ? 2 * stage : red;
}

// One output tile of a product (`tile` from split_slice), LDS at `smem`.
template <typename T, typename TO, bool AK, bool BKM, int BM, int BN, int WM, int WN, int WK,
          int KSEG, bool VA, bool VB, int EPI, bool PH2 = false>
__device__ __forceinline__ void gemm_tile(Params& p, const int tile, char* smem) {
  constexpr int THREADS = 64 * WM * WN * WK;
  constexpr int BK = Elem<T>::BK;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(TM >= 1 && TN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
  static_assert(WK == 1 || WK == 2 || WK == 4, "k-step groups");
  constexpr int SEG = (BM + BN) * kRowStride;        // one k-segment of A and B rows
  constexpr int STAGE = KSEG * SEG;                   // one pipeline stage
  constexpr int KSTAGE = KSEG * BK;                   // k elements per stage

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wk = wave / (WM * WN);          // k-step group
  const int wmn = wave % (WM * WN);
  const int wm = wmn / WN, wn = wmn % WN;

  int tm, tn;
  tile_of(tile, p.tiles_m, p.tiles_n, tm, tn);
  const int64_t m0 = static_cast<int64_t>(tm) * BM;
  const int64_t n0 = static_cast<int64_t>(tn) * BN;

  const T* __restrict__ A = static_cast<const T*>(p.A);
  const T* __restrict__ B = static_cast<const T*>(p.B);

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Bias-gradient column sums (TN): the first row of tiles sums its B tiles.
  constexpr int CS_PER = (BN + THREADS - 1) / THREADS;
  float csum[CS_PER];
#pragma unroll
  for (int i = 0; i < CS_PER; ++i) csum[i] = 0.0f;
  const bool do_colsum = (EPI == EPI_DW) && (p.colsum != nullptr) && (tm == 0);

  TileLoader<T, AK, BM, THREADS, VA, KSEG> la;
  TileLoader<T, BKM, BN, THREADS, VB, KSEG> lb;
  const int64_t nk1 = PH2 ? (p.K1 + KSTAGE - 1) / KSTAGE : (p.K + KSTAGE - 1) / KSTAGE;
  const int64_t nk = PH2 ? nk1 + (p.K - p.K1 + KSTAGE - 1) / KSTAGE : nk1;
  auto load_stage = [&](int64_t kt) {
    const StageSrc<T, BKM> q = stage_src<T, BKM, PH2>(p, A, B, kt, nk1, KSTAGE);
    la.load(q.a, q.lda, m0, p.M, q.k0, q.klim, tid);
    lb.load(q.b, p.ldb, n0, p.N, q.k0, q.klim, tid);
  };

  load_stage(0);
  la.template store<SEG>(smem, tid);
  lb.template store<SEG>(smem + BM * kRowStride, tid);
  __syncthreads();

  const int frag_row = lane & 31;
  const int frag_half = lane >> 5;

  for (int64_t kt = 0; kt < nk; ++kt) {
    const int buf = static_cast<int>(kt & 1);
    char* stage = smem + buf * STAGE;
    const bool more = kt + 1 < nk;
    if (more) load_stage(kt + 1);
#pragma unroll
    for (int g = 0; g < 4 * KSEG; ++g) {
      if constexpr (WK > 1) {
        if (g % WK != wk) continue;  // this group's k-steps
      }
      const char* As = stage + (g / 4) * SEG;
      const char* Bs = As + BM * kRowStride;
      const int cofs = (2 * (g % 4) + frag_half) * 16;
      uint4 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const uint4*>(As + (wm * WTM + i * 32 + frag_row) * kRowStride + cofs);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const uint4*>(Bs + (wn * WTN + j * 32 + frag_row) * kRowStride + cofs);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) mfma_frag<T>(acc[i][j], af[i], bfr[j]);
    }
    if constexpr (EPI == EPI_DW) {
      if (do_colsum) {
#pragma unroll
        for (int ci = 0; ci < CS_PER; ++ci) {
          const int r = tid + ci * THREADS;
          if (r < BN) {
#pragma unroll
            for (int c = 0; c < kChunks * KSEG; ++c) {
              const uint4 x = *reinterpret_cast<const uint4*>(
                  stage + (c / kChunks) * SEG + BM * kRowStride + r * kRowStride + (c % kChunks) * 16);
              const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                if constexpr (sizeof(T) == 4) {
                  csum[ci] += __uint_as_float(w[e]);
                } else {
                  csum[ci] += __uint_as_float(w[e] << 16);
                  csum[ci] += __uint_as_float(w[e] & 0xffff0000u);
                }
              }
            }
          }
        }
      }
    }
    if (more) {
      char* next = smem + (buf ^ 1) * STAGE;
      la.template store<SEG>(next, tid);
      lb.template store<SEG>(next + BM * kRowStride, tid);
    }
    __syncthreads();
  }

  if constexpr (WK > 1) {
    // Add the k-step groups' accumulators through LDS, group 1 first.
    constexpr int WAVE_F = TM * TN * 16 * 64;  // accumulator floats of one wave
    float* red = reinterpret_cast<float*>(smem);
    if (wk > 0) {
      float* dst = red + ((wk - 1) * (WM * WN) + wmn) * WAVE_F;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((i * TN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (wk > 0) {
      // Only the first group runs the epilogue; the column sums (kept by
      // every thread of the workgroup) are written by their owners below.
      if constexpr (EPI == EPI_DW) {
        if (do_colsum) {
#pragma unroll
          for (int ci = 0; ci < CS_PER; ++ci) {
            const int r = tid + ci * THREADS;
            if (r < BN && n0 + r < p.nvec) p.colsum[n0 + r] = csum[ci];
          }
        }
      }
      return;
    }
#pragma unroll
    for (int q = 1; q < WK; ++q) {
      const float* src = red + ((q - 1) * (WM * WN) + wmn) * WAVE_F;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] += src[((i * TN + j) * 16 + r) * 64 + lane];
    }
  }

  // Epilogue.
  if constexpr (EPI == EPI_CHAIN) {
    // Each wavefront's e^2 sum (fixed-order butterfly) is one loss partial:
    // no synchronisation between the wavefronts of the tile.
    float sq = 0.0f;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int i = 0; i < TM; ++i)
        sq += chain_block(p, acc[i][j], m0 + wm * WTM + i * 32, n0 + wn * WTN + j * 32, lane);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sq += __shfl_xor(sq, o, 64);
    if (lane == 0) p.partials[static_cast<int64_t>(tile) * (WM * WN) + wmn] = sq;
    return;
  }
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int i = 0; i < TM; ++i)
      store_block<T, TO, EPI>(p, acc[i][j], m0 + wm * WTM + i * 32, n0 + wn * WTN + j * 32, lane);
  if constexpr (EPI == EPI_DW) {
    if (do_colsum) {
#pragma unroll
      for (int ci = 0; ci < CS_PER; ++ci) {
        const int r = tid + ci * THREADS;
        if (r < BN && n0 + r < p.nvec) p.colsum[n0 + r] = csum[ci];
      }
    }
  }
}

template <typename T, typename TO, bool AK, bool BKM, int BM, int BN, int WM, int WN, int WK,
          int KSEG, bool VA, bool VB, int EPI, bool PH2>
__global__ __launch_bounds__(64 * WM * WN * WK) void dlvm_gemm_kernel(Params p) {
  __shared__ __attribute__((aligned(16))) char smem[gemm_smem_bytes<T, BM, BN, WK, KSEG>()];
  const int tile = split_slice<T, AK, BKM>(p, static_cast<int>(blockIdx.x));
  // a k-slice of a split two-phase product lies in one phase
  if (PH2 && p.splits <= 1)
    gemm_tile<T, TO, AK, BKM, BM, BN, WM, WN, WK, KSEG, VA, VB, EPI, PH2>(p, tile, smem);
  else
    gemm_tile<T, TO, AK, BKM, BM, BN, WM, WN, WK, KSEG, VA, VB, EPI, false>(p, tile, smem);
}

// The two adjoint products of one dense layer in one launch: blocks
// [0, n1) are tiles of the product wrt the weights (TN, float32 dW and the
// bias-gradient column sums), the rest tiles of the product wrt the input
// (NT, activation-derivative epilogue). Both read the same adjoint dY; they
// share nothing else, so the only change is one launch instead of two.
template <typename T, typename TO2, int BM, int BN, int WM, int WN, int WK, int KSEG>
__global__ __launch_bounds__(64 * WM * WN * WK) void dlvm_gemm_pair_kernel(Params p1, Params p2,
                                                                           int n1) {
  __shared__ __attribute__((aligned(16))) char smem[gemm_smem_bytes<T, BM, BN, WK, KSEG>()];
  const int b = static_cast<int>(blockIdx.x);
  if (b < n1) {
    const int tile = split_slice<T, false, false>(p1, b);
    gemm_tile<T, float, false, false, BM, BN, WM, WN, WK, KSEG, true, true, EPI_DW>(p1, tile, smem);
  } else {
    const int tile = split_slice<T, true, true>(p2, b - n1);
    gemm_tile<T, TO2, true, true, BM, BN, WM, WN, WK, KSEG, true, true, EPI_DACT>(p2, tile, smem);
  }
}

// Tile configurations: (BM, BN, waves along M, waves along N, k-step groups,
// k-segments per stage). A stage is KSEG * 128 bytes of k per row.
//   0: 128 x 128, 2 x 2 waves,             1 segment    large products
//   1:  64 x  64, 2 x 2 waves,             2 segments   medium products
//   2: 128 x  32, 4 x 1 waves,             2 segments   narrow outputs (N <= 32)
//   3:  32 x  32, 1 wave x 4 k-groups,     4 segments   small products (latency-bound)
//   4:  64 x  64, 2 x 2 waves x 2 k-groups, 2 segments  (512 threads) medium-small products
template <typename T, typename TO, bool AK, bool BKM, bool VA, bool VB, int EPI, bool PH2 = false>
hipError_t launch_cfg(const Params& p, int cfg, unsigned grid, hipStream_t s) {
  switch (cfg) {
    case 0:
      launch_kernel((dlvm_gemm_kernel<T, TO, AK, BKM, 128, 128, 2, 2, 1, 1, VA, VB, EPI, PH2>), dim3(grid), dim3(256), s, p);
      break;
    case 1:
      launch_kernel((dlvm_gemm_kernel<T, TO, AK, BKM, 64, 64, 2, 2, 1, 2, VA, VB, EPI, PH2>), dim3(grid), dim3(256), s, p);
      break;
    case 2:
      launch_kernel((dlvm_gemm_kernel<T, TO, AK, BKM, 128, 32, 4, 1, 1, 2, VA, VB, EPI, PH2>), dim3(grid), dim3(256), s, p);
      break;
    case 3:
      launch_kernel((dlvm_gemm_kernel<T, TO, AK, BKM, 32, 32, 1, 1, 4, 4, VA, VB, EPI, PH2>), dim3(grid), dim3(256), s, p);
      break;
    case 5:
      launch_kernel((dlvm_gemm_kernel<T, TO, AK, BKM, 32, 32, 1, 1, 4, 8, VA, VB, EPI, PH2>), dim3(grid), dim3(256), s, p);
      break;
    default:
      launch_kernel((dlvm_gemm_kernel<T, TO, AK, BKM, 64, 64, 2, 2, 2, 2, VA, VB, EPI, PH2>), dim3(grid), dim3(512), s, p);
      break;
  }
  return hipGetLastError();
}

template <typename T, typename TO, bool AK, bool BKM, int EPI, bool PH2 = false>
hipError_t launch_vec(const Params& p, int cfg, unsigned grid, bool va, bool vb, hipStream_t s) {
  if (va) {
    return vb ? launch_cfg<T, TO, AK, BKM, true, true, EPI, PH2>(p, cfg, grid, s)
              : launch_cfg<T, TO, AK, BKM, true, false, EPI, PH2>(p, cfg, grid, s);
  }
  return vb ? launch_cfg<T, TO, AK, BKM, false, true, EPI, PH2>(p, cfg, grid, s)
            : launch_cfg<T, TO, AK, BKM, false, false, EPI, PH2>(p, cfg, grid, s);
}

// The two adjoint products of a layer (TN wrt the weights, NT wrt the input)
// in one launch, for the configurations pair_config accepts.
bool pair_config(int dtype, int cfg);
hipError_t launch_pair(const Params& p1, const Params& p2, int n1, unsigned grid, int dtype,
                       int out_dtype2, int cfg, hipStream_t s);

// Per-layout entry points (one translation unit each).
hipError_t launch_nn(const Params& p, int dtype, int out_dtype, int cfg, unsigned grid, bool va,
                     bool vb, hipStream_t s);
hipError_t launch_nt(const Params& p, int dtype, int out_dtype, int cfg, unsigned grid, bool va,
                     bool vb, hipStream_t s);
hipError_t launch_tn(const Params& p, int dtype, int cfg, unsigned grid, bool va, bool vb,
                     hipStream_t s);

}  // namespace gemm
}  // namespace dlvm
