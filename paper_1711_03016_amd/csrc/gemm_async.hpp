// bf16 dense-layer products with asynchronous direct-to-LDS loads and an LDS
// ring of STAGES k-tiles.
//
// Same products and fused epilogues as gemm_kernel.hpp (NN forward, NT adjoint
// wrt the input, TN adjoint wrt the weights), for bf16 operands with 16-byte
// aligned rows (every leading dimension and K a multiple of 8). Differences:
//
// * Global -> LDS with global_load_lds_dwordx4: one wave instruction moves
//   64 x 16 bytes into one contiguous kilobyte of LDS without passing through
//   registers, so several k-tiles are in flight while the matrix cores work on
//   an earlier one. Each lane picks which 16-byte chunk of the operand it
//   fetches so that the contiguous kilobyte holds the swizzled layout below.
// * LDS layouts (no padding). A k-contiguous operand tile is ROWS rows of 128
//   bytes (64 k); the 16-byte chunk c of row r sits in slot c ^ h(r). An
//   m-contiguous (or n-contiguous) tile is 64 k-rows of 2*ROWS bytes; its
//   32-byte column group g of k-row k sits in group g ^ f(k & 3). h and f make
//   the fragment reads below free of bank conflicts whether the LDS serves 128
//   or 256 bytes per clock.
// * Fragments. A k-contiguous operand gives each lane its 8 consecutive k in
//   one 16-byte LDS read. An m-contiguous operand is read with the transposing
//   ds_read_b64_tr_b16: inside a group of 16 lanes, lane r points at 4
//   consecutive elements (columns 4(r%4) .. 4(r%4)+3) of k-row r/4 and lane i
//   receives the 4 k values of column i; two such reads give the 8 k of a
//   fragment. The transposes of the adjoint products are thus done by the LDS
//   read, not by registers and not in memory.
// * Ragged edges. Rows or columns past M or N are loaded from a clamped valid
//   address (they only reach outputs that are not stored). k past K is loaded
//   from a clamped address and then zeroed in LDS before the last k-tile is
//   multiplied.
// * Tile order: tile_of (gemm_kernel.hpp), XCD-aware.
#pragma once

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "gemm_kernel.hpp"

namespace dlvm {
namespace gemm {

typedef short v4i16 __attribute__((ext_vector_type(4)));
#define DLVM_LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

// Swizzle of a k-contiguous tile row: the 16-byte chunk c of row r sits in
// slot c ^ kswz(r). Rows of 128 bytes (BK = 64) have 8 slots, rows of 64 bytes
// (BK = 32) have 4.
template <int BK>
__device__ __forceinline__ int kswz(int r) {
  if constexpr (BK == 64) return (r ^ (r >> 3)) & 7;
  else return ((r >> 1) ^ (r >> 3)) & 3;
}
// Byte offset of 16-byte chunk c of row r in a k-contiguous tile.
template <int BK>
__device__ __forceinline__ int kmaj_off(int r, int c) {
  return r * (2 * BK) + ((c ^ kswz<BK>(r)) << 4);
}
// Byte offset of 16-byte chunk c of k-row k in an m-contiguous tile of RB-byte rows.
template <int RB>
__device__ __forceinline__ int mmaj_off(int k, int c) {
  const int q = k & 3;
  return k * RB + ((c ^ ((q ^ ((q & 1) << 2)) << 1)) << 4);
}

// Element offset (from the operand base) of the 16-byte chunk that lane `lane`
// of wave instruction `kb` fetches for the k-tile starting at k0. Rows past
// rlim and k past klim are clamped to valid addresses.
template <bool KMAJ, int ROWS, int BK>
__device__ __forceinline__ int64_t chunk_src(int kb, int lane, int64_t ld, int64_t r0, int64_t rlim,
                                             int64_t k0, int64_t klim) {
  const int b = kb * 1024 + lane * 16;  // byte of this lane inside the tile
  if constexpr (KMAJ) {
    constexpr int RBK = 2 * BK;
    const int r = b / RBK;
    const int c = ((b % RBK) >> 4) ^ kswz<BK>(r);
    int64_t gr = r0 + r;
    int64_t gk = k0 + c * 8;
    gr = gr < rlim ? gr : rlim - 1;
    gk = gk < klim ? gk : 0;
    return gr * ld + gk;
  } else {
    constexpr int RB = ROWS * 2;
    const int k = b / RB;
    const int q = k & 3;
    const int c = ((b % RB) >> 4) ^ ((q ^ ((q & 1) << 2)) << 1);
    int64_t gk = k0 + k;
    int64_t gr = r0 + c * 8;
    gk = gk < klim ? gk : k0;
    gr = gr < rlim ? gr : 0;
    return gk * ld + gr;
  }
}

// Buffer descriptor of `bytes` bytes at `base` (raw buffer, no swizzle, no
// index stride; the third word is the data-format word of gfx9 raw buffers).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes),
                                           0x00020000);
}

// Byte offsets (k-tile 0) of the 16-byte chunks that lane `lane` of `wave`
// fetches for its LOADS wave instructions of one ROWS x BK operand tile (the
// same chunks as chunk_src, without clamping). KMAJ: rows of BK k (2 BK
// bytes); the chunk c of row r holds k 8c..8c+7 and sits in slot c ^ kswz(r).
// !KMAJ: k-rows of ROWS elements (2 ROWS bytes); the 16-byte column group c of
// k-row k sits in slot c ^ f(k & 3).
template <bool KMAJ, int ROWS, int BK, int LOADS>
__device__ __forceinline__ void tile_offsets(uint32_t (&off)[LOADS], int wave, int lane, int64_t ld,
                                             int64_t r0) {
  constexpr int RB = ROWS * 2;
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int b = (wave * LOADS + j) * 1024 + lane * 16;  // byte inside the tile
    if constexpr (KMAJ) {
      const int r = b / (2 * BK);
      const int c = ((b % (2 * BK)) >> 4) ^ kswz<BK>(r);
      off[j] = static_cast<uint32_t>(((r0 + r) * ld + c * 8) * 2);
    } else {
      const int k = b / RB;
      const int q = k & 3;
      const int c = ((b % RB) >> 4) ^ ((q ^ ((q & 1) << 2)) << 1);
      off[j] = static_cast<uint32_t>((k * ld + r0 + c * 8) * 2);
    }
  }
}
template <bool KMAJ, int BK, int LOADS>
__device__ __forceinline__ void xl_offsets(uint32_t (&off)[LOADS], int wave, int lane, int64_t ld,
                                           int64_t r0) {
  tile_offsets<KMAJ, 256, BK, LOADS>(off, wave, lane, ld, r0);
}

template <bool KMAJ, int ROWS, int BK, int NWAVES>
__device__ __forceinline__ void async_tile(const bf16_t* __restrict__ P, int64_t ld, int64_t r0,
                                           int64_t rlim, int64_t k0, int64_t klim, char* lds,
                                           int wave, int lane) {
  constexpr int KB = ROWS * 2 * BK / 1024;  // wave instructions per tile
  static_assert(KB % NWAVES == 0, "tile split over waves");
#pragma unroll
  for (int j = 0; j < KB / NWAVES; ++j) {
    const int kb = wave * (KB / NWAVES) + j;
    const bf16_t* src = P + chunk_src<KMAJ, ROWS, BK>(kb, lane, ld, r0, rlim, k0, klim);
    __builtin_amdgcn_global_load_lds(src, DLVM_LDS_PTR(lds + kb * 1024), 16, 0, 0);
  }
}

// Zero the k >= kv part of a tile (last k-tile of a ragged K; kv % 8 == 0).
template <bool KMAJ, int ROWS, int BK, int THREADS>
__device__ __forceinline__ void zero_k_tail(char* lds, int kv, int tid) {
  const uint4 z = make_uint4(0u, 0u, 0u, 0u);
  if constexpr (KMAJ) {
    constexpr int KC = BK / 8;
    for (int q = tid; q < ROWS * KC; q += THREADS) {
      const int r = q / KC, c = q % KC;
      if (c * 8 >= kv) *reinterpret_cast<uint4*>(lds + kmaj_off<BK>(r, c)) = z;
    }
  } else {
    constexpr int RB = ROWS * 2;
    for (int q = kv * (RB / 16) + tid; q < BK * (RB / 16); q += THREADS)
      *reinterpret_cast<uint4*>(lds + q * 16) = z;  // whole k-rows: the swizzle does not matter
  }
}

// Fragment (8 k per lane) of the 32-row block at `row0` for k-step s (16 k).
template <bool KMAJ, int ROWS, int BK>
__device__ __forceinline__ bf16x8 frag(const char* lds, int row0, int s, int lane) {
  if constexpr (KMAJ) {
    const int r = row0 + (lane & 31);
    const int c = 2 * s + (lane >> 5);
    return *reinterpret_cast<const bf16x8*>(lds + kmaj_off<BK>(r, c));
  } else {
    constexpr int RB = ROWS * 2;
    const int g = lane >> 4, r = lane & 15;
    const int col = row0 + 16 * (g & 1) + 4 * (r & 3);
    const int k = 16 * s + 8 * (g >> 1) + (r >> 2);
    const int in16 = (col & 7) * 2;
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4i16*)(lds + mmaj_off<RB>(k, col >> 3) + in16));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4i16*)(lds + mmaj_off<RB>(k + 4, col >> 3) + in16));
    const v4i16 v8[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, v8);
  }
}

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
template <int LOADS, int MAXA>
__device__ __forceinline__ void wait_stage(int ahead) {
  if constexpr (MAXA >= 3) { if (ahead >= 3) { wait_vm<3 * LOADS>(); return; } }
  if constexpr (MAXA >= 2) { if (ahead == 2) { wait_vm<2 * LOADS>(); return; } }
  if constexpr (MAXA >= 1) { if (ahead == 1) { wait_vm<LOADS>(); return; } }
  wait_vm<0>();
}

// Barrier between the waves of the workgroup that waits for nothing itself
// (the callers wait for exactly what must have landed), plus a compiler-only
// fence so that no LDS access is moved across it.
__device__ __forceinline__ void barrier_only() {
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// One k-tile (BK k) of the wave's TM x TN blocks of 32 x 32, the fragments of
// the next 16 k read while the matrix cores work on the current ones. The
// operand tiles come in through restrict parameters: the LDS reads then carry
// alias-scope information, which tells the compiler that they do not depend on
// the direct-to-LDS loads in flight into the other ring slots (the explicit
// waits and barriers order the slot being read).
//
// With CS and do_cs, cs[j] also accumulates the B fragments of block column j:
// lane l adds the 8 k values it holds of column l % 32, so that over all
// k-tiles the two halves of the wave (lanes l and l + 32) hold complementary
// partial column sums of B.
// ILV > 0: instead of keeping all of a step's fragment reads ahead of its
// matrix instructions, the scheduler is asked to alternate them, one matrix
// instruction then (ILV & 7) LDS reads (ILV >= 8 also raises the wave's issue
// priority around the matrix instructions). Measured on the 16384 x 4096 x
// 4096 products of the deep bf16 network (256 x 256 tiles): ILV 4 about 2%
// faster than the reads kept ahead; priority no gain.
template <bool AK, bool BKM, int BM, int BN, int BK, int TM, int TN, bool CS, int ILV = 0>
__device__ __forceinline__ void mma_ktile(const char* __restrict__ As, const char* __restrict__ Bs,
                                          int arow, int brow, int lane, f32x16 (&acc)[TM][TN],
                                          float (&cs)[TN], bool do_cs) {
  constexpr int S = BK / 16;
  bf16x8 af[2][TM], bfr[2][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) af[0][i] = frag<AK, BM, BK>(As, arow + i * 32, 0, lane);
#pragma unroll
  for (int j = 0; j < TN; ++j) bfr[0][j] = frag<BKM, BN, BK>(Bs, brow + j * 32, 0, lane);
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int cur = s & 1, nxt = cur ^ 1;
    if (s + 1 < S) {
#pragma unroll
      for (int i = 0; i < TM; ++i) af[nxt][i] = frag<AK, BM, BK>(As, arow + i * 32, s + 1, lane);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[nxt][j] = frag<BKM, BN, BK>(Bs, brow + j * 32, s + 1, lane);
    }
    // The next step's fragment reads stay ahead of this step's matrix
    // instructions (otherwise the scheduler waits on each read in turn).
    if constexpr (ILV == 0) __builtin_amdgcn_sched_barrier(0);
    if constexpr (ILV >= 8) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
    if constexpr (ILV > 0) {
#pragma unroll
      for (int q = 0; q < TM * TN; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);         // one matrix instruction
        __builtin_amdgcn_sched_group_barrier(0x100, ILV & 7, 0);   // then (ILV & 7) LDS reads
      }
    }
    if constexpr (ILV >= 8) __builtin_amdgcn_s_setprio(0);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (CS) {
      if (do_cs) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const uint4 w = __builtin_bit_cast(uint4, bfr[cur][j]);
          const uint32_t q[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            cs[j] += __uint_as_float(q[e] << 16);
            cs[j] += __uint_as_float(q[e] & 0xffff0000u);
          }
        }
      }
    }
  }
}

// NS consecutive 16-k steps of a k-tile from step s0 (a tile whose waves form
// k-groups gives each group its own steps of every k-tile), the next step's
// fragments read while the matrix cores work on the current ones; with CS and
// do_cs, the column sums of the B fragments as in mma_ktile.
template <bool AK, bool BKM, int BM, int BN, int BK, int TM, int TN, int NS, bool CS>
__device__ __forceinline__ void mma_ksteps(const char* __restrict__ As, const char* __restrict__ Bs,
                                           int s0, int arow, int brow, int lane,
                                           f32x16 (&acc)[TM][TN], float (&cs)[TN], bool do_cs) {
  bf16x8 af[2][TM], bfr[2][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) af[0][i] = frag<AK, BM, BK>(As, arow + i * 32, s0, lane);
#pragma unroll
  for (int j = 0; j < TN; ++j) bfr[0][j] = frag<BKM, BN, BK>(Bs, brow + j * 32, s0, lane);
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int cur = s & 1, nxt = cur ^ 1;
    if (s + 1 < NS) {
#pragma unroll
      for (int i = 0; i < TM; ++i) af[nxt][i] = frag<AK, BM, BK>(As, arow + i * 32, s0 + s + 1, lane);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[nxt][j] = frag<BKM, BN, BK>(Bs, brow + j * 32, s0 + s + 1, lane);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (CS) {
      if (do_cs) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const uint4 w = __builtin_bit_cast(uint4, bfr[cur][j]);
          const uint32_t q[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            cs[j] += __uint_as_float(q[e] << 16);
            cs[j] += __uint_as_float(q[e] & 0xffff0000u);
          }
        }
      }
    }
  }
}

// Partial sums of block rows [I0, I0 + TH) of a wave's accumulators to LDS
// (xchg_put), or added from LDS (xchg_add): TH x TN blocks as 4 float4 per
// lane each, lane-interleaved (lane l's float4 q at xb[(slot + q) * 64 + l]).
template <int I0, int TH, int TM, int TN>
__device__ __forceinline__ void xchg_put(float4* xb, const f32x16 (&acc)[TM][TN], int slot,
                                         int lane) {
#pragma unroll
  for (int i = 0; i < TH; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const f32x16& a = acc[I0 + i][j];
        xb[(slot + (i * TN + j) * 4 + r) * 64 + lane] =
            make_float4(a[4 * r], a[4 * r + 1], a[4 * r + 2], a[4 * r + 3]);
      }
}
template <int I0, int TH, int TM, int TN>
__device__ __forceinline__ void xchg_add(const float4* xb, f32x16 (&acc)[TM][TN], int slot,
                                         int lane) {
#pragma unroll
  for (int i = 0; i < TH; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float4 v = xb[(slot + (i * TN + j) * 4 + r) * 64 + lane];
        acc[I0 + i][j][4 * r] += v.x;
        acc[I0 + i][j][4 * r + 1] += v.y;
        acc[I0 + i][j][4 * r + 2] += v.z;
        acc[I0 + i][j][4 * r + 3] += v.w;
      }
}

// Vector access to 8 consecutive elements (16 bytes of bf16, 32 of float32).
__device__ __forceinline__ void load8(const bf16_t* p, float (&v)[8]) {
  const uint4 w = *reinterpret_cast<const uint4*>(p);
  const uint32_t q[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[2 * e] = __uint_as_float(q[e] << 16);
    v[2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void store8(bf16_t* p, const float (&v)[8]) {
  uint32_t q[4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    q[e] = static_cast<uint32_t>(f32_to_bf16(v[2 * e])) |
           (static_cast<uint32_t>(f32_to_bf16(v[2 * e + 1])) << 16);
  *reinterpret_cast<uint4*>(p) = make_uint4(q[0], q[1], q[2], q[3]);
}
__device__ __forceinline__ void store8(float* p, const float (&v)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

// Rectifier masks (Params::mask; the host sets one only with the rectifier,
// which these two functions assume). The forward product of a rectified layer
// stores its 32 x 32 blocks as store_block does and keeps, per element, the
// bit (stored output > 0), which is the rectifier's derivative taken from the
// saved output; the adjoint product of the next layer has the same tile and
// wave decomposition of the same output shape, so lane t of its workgroup
// holds the same elements and reads its 128 bits as one 16-byte word instead
// of 256 bytes of saved activation through LDS.
__device__ __forceinline__ uint32_t store_block_bits(const Params& p, const f32x16& acc,
                                                     int64_t r0, int64_t c0, int lane) {
  const int64_t col = c0 + (lane & 31);
  const int64_t rb = r0 + 4 * (lane >> 5);
  const bool full = r0 + 32 <= p.M && c0 + 32 <= p.N;
  const int ld = static_cast<int>(p.ldc);
  float bias_v = 0.0f;
  if (p.bias != nullptr && col < p.nvec) bias_v = bf16_to_f32(static_cast<const bf16_t*>(p.bias)[col]);
  bf16_t* __restrict__ C = static_cast<bf16_t*>(p.C) + rb * p.ldc + col;
  uint32_t bits = 0;
  auto one = [&](int r) {
    const int ro = 8 * (r >> 2) + (r & 3);
    const float z = p.alpha * acc[r] + bias_v;
    const bf16_t o = f32_to_bf16(z > 0.0f ? z : 0.0f);  // apply_act(ACT_RELU, z)
    C[ro * ld] = o;
    bits |= (bf16_to_f32(o) > 0.0f ? 1u : 0u) << r;  // act_grad_from_output(ACT_RELU, o) > 0
  };
  if (full) {
#pragma unroll
    for (int r = 0; r < 16; ++r) one(r);
  } else if (col < p.N) {
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (rb + 8 * (r >> 2) + (r & 3) < p.M) one(r);
  }
  return bits;
}

// The adjoint's store of one block with the rectifier's derivative from the
// block's 16 mask bits: the same arithmetic as the saved-activation path
// without a residual (product times derivative, plus a zero residual).
template <typename TO>
__device__ __forceinline__ void store_block_masked(const Params& p, const f32x16& acc, int64_t r0,
                                                   int64_t c0, int lane, uint32_t bits) {
  const int64_t col = c0 + (lane & 31);
  const int64_t rb = r0 + 4 * (lane >> 5);
  const bool full = r0 + 32 <= p.M && c0 + 32 <= p.N;
  const int ld = static_cast<int>(p.ldc);
  TO* __restrict__ C = static_cast<TO*>(p.C) + rb * p.ldc + col;
  auto one = [&](int r) {
    const float d = ((bits >> r) & 1u) ? 1.0f : 0.0f;
    C[(8 * (r >> 2) + (r & 3)) * ld] = store_cast<TO>(acc[r] * d + 0.0f);
  };
  if (full) {
#pragma unroll
    for (int r = 0; r < 16; ++r) one(r);
  } else if (col < p.N) {
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (rb + 8 * (r >> 2) + (r & 3) < p.M) one(r);
  }
}

// Epilogue of one row of a wave's 32 x 32 accumulator blocks (32 x WTN
// outputs starting at (r0, c0)) through the wave's own LDS region: the
// accumulators are written to LDS in row-major order, then every lane takes
// chunks of 8 consecutive columns of one row, so the saved activation,
// residual, bias and output move as 16-byte (bf16) or 32-byte (float32)
// vectors, 8 lanes covering a row segment of WTN columns. Chunks that cross
// the output's edge are done element by element. Requires ldc % 8 == 0 and
// 16-byte aligned C, aux, residual and bias.
template <typename TO, int EPI, int TN>
__device__ __forceinline__ void epilogue_row(const Params& p, const f32x16 (&acc)[TN],
                                             float* region, int64_t r0, int64_t c0, int lane) {
  constexpr int WTN = TN * 32;
  constexpr int LDF = WTN + 4;         // floats per LDS row (padding spreads the banks)
  constexpr int CPR = WTN / 8;         // chunks per row
  constexpr int CPL = 32 * CPR / 64;   // chunks per lane
  constexpr int BATCH = 2;             // chunks whose loads are in flight together
  static_assert(CPL % BATCH == 0, "chunk batches");
  TO* __restrict__ C = static_cast<TO*>(p.C);
  const bf16_t* __restrict__ aux = static_cast<const bf16_t*>(p.aux);
  const TO* __restrict__ res = static_cast<const TO*>(p.residual);
  const bf16_t* __restrict__ bias = static_cast<const bf16_t*>(p.bias);
  const bool has_act = p.act != ACT_NONE;
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      region[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * LDF + j * 32 + (lane & 31)] = acc[j][r];
  // The rows are read back by other lanes of the same wave: wait for the
  // writes, and keep the compiler from moving the reads above them.
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  for (int t0 = 0; t0 < CPL; t0 += BATCH) {
    float x[BATCH][8], g[BATCH][8], rv[BATCH][8];
    int64_t row[BATCH], col[BATCH];
    bool full[BATCH];
#pragma unroll
    for (int b = 0; b < BATCH; ++b) {
      const int q = lane + 64 * (t0 + b);
      const int rr = q / CPR, cc = (q % CPR) * 8;
      row[b] = r0 + rr;
      col[b] = c0 + cc;
      full[b] = row[b] < p.M && col[b] + 8 <= p.N;
      const float4 lo = *reinterpret_cast<const float4*>(region + rr * LDF + cc);
      const float4 hi = *reinterpret_cast<const float4*>(region + rr * LDF + cc + 4);
      x[b][0] = lo.x; x[b][1] = lo.y; x[b][2] = lo.z; x[b][3] = lo.w;
      x[b][4] = hi.x; x[b][5] = hi.y; x[b][6] = hi.z; x[b][7] = hi.w;
      const int64_t idx = row[b] * p.ldc + col[b];
#pragma unroll
      for (int e = 0; e < 8; ++e) { g[b][e] = 0.0f; rv[b][e] = 0.0f; }
      if constexpr (EPI == EPI_STORE) {
        if (bias != nullptr) {
          if (col[b] + 8 <= p.nvec) {
            load8(bias + col[b], g[b]);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (col[b] + e < p.nvec) g[b][e] = bf16_to_f32(bias[col[b] + e]);
          }
        }
      } else if constexpr (EPI == EPI_DACT) {
        if (full[b]) {
          if (has_act) load8(aux + idx, g[b]);
          if (res != nullptr) load8(res + idx, rv[b]);
        } else if (row[b] < p.M) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if (col[b] + e < p.N) {
              if (has_act) g[b][e] = bf16_to_f32(aux[idx + e]);
              if (res != nullptr) rv[b][e] = load_as_f32<TO>(res + idx + e);
            }
          }
        }
      }
    }
#pragma unroll
    for (int b = 0; b < BATCH; ++b) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[e] = x[b][e];
        if constexpr (EPI == EPI_STORE) {
          v[e] = apply_act(p.act, p.alpha * v[e] + g[b][e]);
        } else if constexpr (EPI == EPI_DACT) {
          if (p.res_pre) v[e] += rv[b][e];
          if (has_act) v[e] *= act_grad_from_output(p.act, g[b][e]);
          if (!p.res_pre) v[e] += rv[b][e];
        }
      }
      const int64_t idx = row[b] * p.ldc + col[b];
      if (full[b]) {
        store8(C + idx, v);
      } else if (row[b] < p.M) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (col[b] + e < p.N) C[idx + e] = store_cast<TO>(v[e]);
      }
    }
  }
  // The region is written again for the next row: keep its reads above.
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Rows of blocks [I, IEND) (all TM by default), each with a statically
// indexed accumulator row; r0 is the row of block row 0.
template <typename TO, int EPI, int TM, int TN, int I = 0, int IEND = TM>
__device__ __forceinline__ void epilogue_lds(const Params& p, const f32x16 (&acc)[TM][TN],
                                             float* region, int64_t r0, int64_t c0, int lane) {
  if constexpr (I < IEND) {
    epilogue_row<TO, EPI, TN>(p, acc[I], region, r0 + 32 * I, c0, lane);
    epilogue_lds<TO, EPI, TM, TN, I + 1, IEND>(p, acc, region, r0, c0, lane);
  }
}

// Zero k >= kv of both operand tiles of a ring slot, then wait for every wave.
template <bool AK, bool BKM, int BM, int BN, int BK, int THREADS, int A_BYTES>
__device__ __forceinline__ void zero_tail_slot(char* slot, int kv, int tid) {
  zero_k_tail<AK, BM, BK, THREADS>(slot, kv, tid);
  zero_k_tail<BKM, BN, BK, THREADS>(slot + A_BYTES, kv, tid);
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the LDS writes are done
  barrier_only();
}

// One 16-k step: the matrix instructions of the fragments in register set
// CUR into acc, the reads of step s2 of the tile at (As2, Bs2) into the other
// set interleaved with them when RD (ILV reads per matrix instruction), and
// the column sums of the step's B fragments.
template <bool AK, bool BKM, int BM, int BN, int BK, int TM, int TN, bool CS, int ILV, bool RD,
          int CUR>
__device__ __forceinline__ void mma_step(bf16x8 (&af)[2][TM], bf16x8 (&bfr)[2][TN],
                                         const char* __restrict__ As2, const char* __restrict__ Bs2,
                                         int s2, int arow, int brow, int lane,
                                         f32x16 (&acc)[TM][TN], float (&cs)[TN], bool do_cs) {
  if constexpr (RD) {
#pragma unroll
    for (int i = 0; i < TM; ++i) af[CUR ^ 1][i] = frag<AK, BM, BK>(As2, arow + i * 32, s2, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[CUR ^ 1][j] = frag<BKM, BN, BK>(Bs2, brow + j * 32, s2, lane);
  }
  if constexpr (ILV == 0) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[CUR][i], bfr[CUR][j], acc[i][j], 0, 0,
                                                          0);
  if constexpr (ILV > 0 && RD) {
#pragma unroll
    for (int q = 0; q < TM * TN; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, ILV & 7, 0);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (CS) {
    if (do_cs) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const uint4 w = __builtin_bit_cast(uint4, bfr[CUR][j]);
        const uint32_t q[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          cs[j] += __uint_as_float(q[e] << 16);
          cs[j] += __uint_as_float(q[e] & 0xffff0000u);
        }
      }
    }
  }
}

// Buffer-descriptor direct loads of k-tile kt of a 256 x 256 tile's A and B
// into ring slot `st`: LA and LB wave instructions per operand, at the lane's
// precomputed byte offsets; the descriptors start at the k-tile's origin
// (kt * step bytes into the operand).
template <int LA, int LB, int A_BYTES>
__device__ __forceinline__ void buf_ktile(const Params& p, int kt, uint32_t stepa, uint32_t stepb,
                                          char* st, const uint32_t* offa, const uint32_t* offb,
                                          int wave) {
  const uint32_t sa = static_cast<uint32_t>(kt) * stepa, sb = static_cast<uint32_t>(kt) * stepb;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(static_cast<const char*>(p.A) + sa, p.a_bytes - sa);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(static_cast<const char*>(p.B) + sb, p.b_bytes - sb);
#pragma unroll
  for (int j = 0; j < LA; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, DLVM_LDS_PTR(st + (wave * LA + j) * 1024), 16,
                                             offa[j], 0, 0, 0);
#pragma unroll
  for (int j = 0; j < LB; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, DLVM_LDS_PTR(st + A_BYTES + (wave * LB + j) * 1024),
                                             16, offb[j], 0, 0, 0);
}

// One output tile (`tile` from split_slice) of the direct-to-LDS kernel, LDS
// ring at `smem` (STAGES * (BM + BN) * 2 * BK bytes, 1024-byte aligned).
// WK = 2: the waves form two k-groups of WM x WN waves over the same output
// blocks, each taking half of every k-tile's 16-k steps (twice the waves per
// SIMD with the LDS reads of WM x WN waves per k-tile); their partial sums are
// added through LDS at the end and each group stores half of the block rows.
template <typename TO, bool AK, bool BKM, int BM, int BN, int BK, int WM, int WN, int STAGES,
          int EPI, bool PH2 = false, int ILV = 0, bool BUFOK = true, bool EARLY = false,
          int WK = 1>
__device__ __forceinline__ void async_gemm_tile(Params& p, const int tile, char* smem) {
  constexpr int NW = WM * WN * WK;
  constexpr int THREADS = 64 * NW;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_BYTES = BM * 2 * BK, B_BYTES = BN * 2 * BK;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int LOADS = STAGE / 1024 / NW;  // direct loads per lane per k-tile
  static_assert(BK == 32 || BK == 64, "k-tile depth");
  static_assert(STAGES >= 2 && STAGES - 2 <= 3 && 3 * LOADS < 64, "pipeline depth");
  static_assert(AK || BM >= 128, "m-contiguous tile needs 256-byte k-rows");
  static_assert(BKM || BN >= 128, "n-contiguous tile needs 256-byte k-rows");
  static_assert(WK == 1 || (WK == 2 && !EARLY && TM % 2 == 0 && BK == 64),
                "k-groups: two, without the early barrier");

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wk = wave / (WM * WN);  // k-group
  const int wm = (wave % (WM * WN)) / WN, wn = wave % WN;
  int tm, tn;
  tile_of(tile, p.tiles_m, p.tiles_n, tm, tn);
  const int64_t m0 = static_cast<int64_t>(tm) * BM;
  const int64_t n0 = static_cast<int64_t>(tn) * BN;
  const bf16_t* __restrict__ A = static_cast<const bf16_t*>(p.A);
  const bf16_t* __restrict__ B = static_cast<const bf16_t*>(p.B);
  // k-tiles of the two phases of the contraction (PH2), else of its one phase
  const int64_t K1 = PH2 ? p.K1 : p.K;
  const int nk1 = static_cast<int>((K1 + BK - 1) / BK);
  const int nk = PH2 ? nk1 + static_cast<int>((p.K - K1 + BK - 1) / BK) : nk1;
  // valid k of the last tile of phase 1 and of phase 2
  const int kv1 = static_cast<int>(K1 - static_cast<int64_t>(nk1 - 1) * BK);
  const int kv2 = PH2 ? static_cast<int>(p.K - K1 - static_cast<int64_t>(nk - nk1 - 1) * BK) : BK;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Bias-gradient column sums (TN): taken from the B fragments by the waves
  // of the first row of tiles that cover the first WTM rows.
  float cs[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) cs[j] = 0.0f;
  const bool do_colsum = (EPI == EPI_DW) && (p.colsum != nullptr) && (tm == 0) && (wm == 0);

  // Rectifier mask (256 x 256 tiles on 2 x 4 waves and 64 x 128 tiles on
  // 2 x 2 waves, one phase, bf16 output): MW words per lane, 16 bits per
  // 32 x 32 block; the adjoint's words are loaded before the contraction so
  // that their latency hides behind it.
  constexpr int MW = TM * TN / 2;
  constexpr bool MASKABLE = ((BM == 256 && BN == 256 && WM == 2 && WN == 4) ||
                             (BM == 64 && BN == 128 && WM == 2 && WN == 2)) &&
                            WK == 1 && !PH2 &&
                            (EPI == EPI_DACT || (EPI == EPI_STORE && std::is_same<TO, bf16_t>::value));
  uint32_t* const mask_word =
      MASKABLE && p.mask != nullptr
          ? p.mask + (static_cast<int64_t>(tm) * p.tiles_n + tn) * (MW * THREADS) + MW * tid
          : nullptr;
  uint32_t mk[MW > 0 ? MW : 1] = {};
  if constexpr (MASKABLE && EPI == EPI_DACT) {
    static_assert(MW == 1 || MW == 4, "one or four mask words per lane");
    if (mask_word != nullptr) {
      if constexpr (MW == 4) {
        const uint4 v = *reinterpret_cast<const uint4*>(mask_word);
        mk[0] = v.x; mk[1] = v.y; mk[2] = v.z; mk[3] = v.w;
      } else {
        mk[0] = *mask_word;
      }
    }
  }

  auto issue = [&](int kt) {
    char* st = smem + (kt % STAGES) * STAGE;
    const StageSrc<bf16_t, BKM> q = stage_src<bf16_t, BKM, PH2>(p, A, B, kt, nk1, BK);
    async_tile<AK, BM, BK, NW>(q.a, q.lda, m0, p.M, q.k0, q.klim, st, wave, lane);
    async_tile<BKM, BN, BK, NW>(q.b, p.ldb, n0, p.N, q.k0, q.klim, st + A_BYTES, wave, lane);
  };

  // Buffer-descriptor loads (one-phase products; the host sets the operand
  // extents a_bytes and b_bytes, below 2^31 bytes, for every such launch).
  // Each lane's byte offsets inside a k-tile are computed once; a k-tile's
  // loads only move the descriptors' base and size (scalar work), and the
  // hardware returns zero for offsets past the size, so rows past M or N need
  // no clamping. Measured on the deep network's 16384 x 4096 x 4096 products
  // (256 x 256 tile): the forward that writes the rectifier mask 540 ->
  // 482-488 us, the input adjoint reading it 476 -> 466-469, the weight
  // adjoint 510 -> 482-485 (the computed addresses cost about 100 vector
  // instructions per wave and k-tile between the barrier and the first matrix
  // instruction); the loads spread over the k-tile's 16-k steps instead were
  // slower than issuing them together. An unsplit two-phase product computes
  // every load's clamped address (issue above), and so does BUFOK = false; a
  // k-slice of a two-phase product lies in one phase and loads through a
  // descriptor of that phase's operand (the host passes both extents).
  constexpr bool BUF = BUFOK && !PH2;
  constexpr int LA = A_BYTES / 1024 / NW, LB = B_BYTES / 1024 / NW;
  uint32_t offa[BUF ? LA : 1], offb[BUF ? LB : 1];
  uint32_t stepa = 0, stepb = 0;
  if constexpr (BUF) {
    tile_offsets<AK, BM, BK, LA>(offa, wave, lane, p.lda, m0);
    tile_offsets<BKM, BN, BK, LB>(offb, wave, lane, p.ldb, n0);
    stepa = AK ? BK * 2 : static_cast<uint32_t>(BK * p.lda * 2);
    stepb = BKM ? BK * 2 : static_cast<uint32_t>(BK * p.ldb * 2);
  }
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s) {
    if (s < nk) {
      if constexpr (BUF)
        buf_ktile<LA, LB, A_BYTES>(p, s, stepa, stepb, smem + s * STAGE, offa, offb, wave);
      else
        issue(s);
    }
  }

  if constexpr (EARLY) {
    // The k-tile's barrier sits before its last 16-k step instead of at its
    // start: the last step's matrix instructions run while the next k-tile's
    // first fragments are read, and the previous step's instructions are
    // still in the matrix pipeline during the wait. Bitwise the same sums.
    static_assert(BUF && STAGES == 2, "early barrier: buffer loads, two stages");
    constexpr int S = BK / 16;
    static_assert(S == 2 || S == 4, "two or four 16-k steps");
    if (nk > 1) buf_ktile<LA, LB, A_BYTES>(p, 1, stepa, stepb, smem + STAGE, offa, offb, wave);
    if (nk > 1) wait_vm<LOADS>();
    else wait_vm<0>();
    barrier_only();
    // (k past K in the last k-tile is zeroed once it has landed, everyone waiting)
    if (nk == 1 && kv1 < BK) zero_tail_slot<AK, BKM, BM, BN, BK, THREADS, A_BYTES>(smem, kv1, tid);
    bf16x8 af[2][TM], bfr[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) af[0][i] = frag<AK, BM, BK>(smem, wm * WTM + i * 32, 0, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j)
      bfr[0][j] = frag<BKM, BN, BK>(smem + A_BYTES, wn * WTN + j * 32, 0, lane);
    for (int kt = 0; kt < nk; ++kt) {
      const char* As = smem + (kt % 2) * STAGE;
      const char* Bs = As + A_BYTES;
      mma_step<AK, BKM, BM, BN, BK, TM, TN, EPI == EPI_DW, ILV, true, 0>(
          af, bfr, As, Bs, 1, wm * WTM, wn * WTN, lane, acc, cs, do_colsum);
      if constexpr (S == 4) {
        mma_step<AK, BKM, BM, BN, BK, TM, TN, EPI == EPI_DW, ILV, true, 1>(
            af, bfr, As, Bs, 2, wm * WTM, wn * WTN, lane, acc, cs, do_colsum);
        mma_step<AK, BKM, BM, BN, BK, TM, TN, EPI == EPI_DW, ILV, true, 0>(
            af, bfr, As, Bs, 3, wm * WTM, wn * WTN, lane, acc, cs, do_colsum);
      }
      // Every read of this k-tile's slot is done (the last step's fragments
      // are in registers) and the next k-tile has landed: then the slot is
      // refilled with k-tile kt + 2 and the next k-tile's first fragments read.
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
      const bool more = kt + 1 < nk;
      if (more) wait_vm<0>();
      barrier_only();
      if (kt + 2 < nk)
        buf_ktile<LA, LB, A_BYTES>(p, kt + 2, stepa, stepb, smem + (kt % 2) * STAGE, offa, offb,
                                   wave);
      constexpr int last = (S - 1) & 1;
      if (more && kt + 1 == nk - 1 && kv1 < BK)
        zero_tail_slot<AK, BKM, BM, BN, BK, THREADS, A_BYTES>(smem + ((kt + 1) % 2) * STAGE, kv1,
                                                             tid);
      // (after the last k-tile these reads of the other slot are not used)
      const char* An = smem + ((kt + 1) % 2) * STAGE;
      mma_step<AK, BKM, BM, BN, BK, TM, TN, EPI == EPI_DW, ILV, true, last>(
          af, bfr, An, An + A_BYTES, 0, wm * WTM, wn * WTN, lane, acc, cs, do_colsum);
    }
  } else
  for (int kt = 0; kt < nk; ++kt) {
    // Stage kt has landed once at most `ahead` later stages are outstanding.
    const int left = nk - 1 - kt;
    wait_stage<LOADS, STAGES - 2>(left < STAGES - 2 ? left : STAGES - 2);
    barrier_only();
    char* As = smem + (kt % STAGES) * STAGE;
    char* Bs = As + A_BYTES;
    const int kv = kt == nk1 - 1 ? kv1 : ((PH2 && kt == nk - 1) ? kv2 : BK);
    if (kv < BK) {
      zero_k_tail<AK, BM, BK, THREADS>(As, kv, tid);
      zero_k_tail<BKM, BN, BK, THREADS>(Bs, kv, tid);
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the LDS writes are done
      barrier_only();
    }
    // The slot refilled here was last read in iteration kt - 1, before the barrier.
    const int kn = kt + STAGES - 1;
    if (kn < nk) {
      if constexpr (BUF)
        buf_ktile<LA, LB, A_BYTES>(p, kn, stepa, stepb, smem + (kn % STAGES) * STAGE, offa, offb,
                                   wave);
      else
        issue(kn);
    }
    if constexpr (WK == 1)
      mma_ktile<AK, BKM, BM, BN, BK, TM, TN, EPI == EPI_DW, ILV>(As, Bs, wm * WTM, wn * WTN, lane,
                                                                 acc, cs, do_colsum);
    else
      mma_ksteps<AK, BKM, BM, BN, BK, TM, TN, BK / 32, EPI == EPI_DW>(
          As, Bs, wk * (BK / 32), wm * WTM, wn * WTN, lane, acc, cs, do_colsum);
  }

  if constexpr (WK == 2) {
    // Group 0 finishes block rows [0, TM/2) of the wave's blocks, group 1 the
    // rest: each first hands the other group its partials of the other half
    // (through LDS, once every wave is done with the ring) and adds the
    // other's partials of its own half (a two-term sum: the same whichever
    // group adds).
    constexpr int TH = TM / 2;
    constexpr int XW = TH * TN * 4;  // float4 per lane handed over
    // (then the column sums of group 1, TN floats per lane of each wave)
    constexpr int XCS = NW * XW * 64 * 16;
    static_assert(XCS + (EPI == EPI_DW ? WM * WN * TN * 64 * 4 : 0) <= STAGES * STAGE,
                  "exchange fits the ring");
    float4* xb = reinterpret_cast<float4*>(smem);
    float* xc = reinterpret_cast<float*>(smem + XCS);
    const int partner = wave ^ (WM * WN);
    barrier_only();
    if (wk == 0)
      xchg_put<TH, TH, TM, TN>(xb, acc, wave * XW, lane);
    else
      xchg_put<0, TH, TM, TN>(xb, acc, wave * XW, lane);
    if constexpr (EPI == EPI_DW) {
      if (do_colsum && wk == 1) {
#pragma unroll
        for (int j = 0; j < TN; ++j) xc[((wave - WM * WN) * TN + j) * 64 + lane] = cs[j];
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the writes are done
    barrier_only();
    if (wk == 0)
      xchg_add<0, TH, TM, TN>(xb, acc, partner * XW, lane);
    else
      xchg_add<TH, TH, TM, TN>(xb, acc, partner * XW, lane);
    if constexpr (EPI == EPI_DW) {
      // group 0 completes the column sums: its partial plus group 1's
      if (do_colsum && wk == 0) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const float t0 = cs[j] + xc[(wave * TN + j) * 64 + lane];
          const float t = t0 + __shfl_xor(t0, 32);
          const int64_t col = n0 + wn * WTN + j * 32 + lane;
          if (lane < 32 && col < p.nvec) p.colsum[col] = t;
        }
      }
    }
    const int64_t rw = m0 + wm * WTM, cw = n0 + wn * WTN;
    if constexpr (EPI == EPI_DACT) {
      static_assert(NW * 32 * (WTN + 4) * 4 <= STAGES * STAGE, "epilogue staging fits the ring");
      __builtin_amdgcn_s_waitcnt(0xc07f);  // the exchange reads are done
      barrier_only();
      float* region = reinterpret_cast<float*>(smem) + wave * 32 * (WTN + 4);
      if (wk == 0)
        epilogue_lds<TO, EPI, TM, TN, 0, TH>(p, acc, region, rw, cw, lane);
      else
        epilogue_lds<TO, EPI, TM, TN, TH, TM>(p, acc, region, rw, cw, lane);
    } else {
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int i = 0; i < TH; ++i) {
          if (wk == 0)
            store_block<bf16_t, TO, EPI>(p, acc[i][j], rw + i * 32, cw + j * 32, lane);
          else
            store_block<bf16_t, TO, EPI>(p, acc[TH + i][j], rw + (TH + i) * 32, cw + j * 32, lane);
        }
    }
    return;
  }

  if (MASKABLE && mask_word != nullptr) {
    if constexpr (MASKABLE) {
      static_assert(MW == 1 || MW == 4, "one or four mask words per lane");
      uint32_t w[MW];
#pragma unroll
      for (int q = 0; q < MW; ++q) w[q] = mk[q];
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int q = i * TN + j;
          const int64_t r0 = m0 + wm * WTM + i * 32, c0 = n0 + wn * WTN + j * 32;
          if constexpr (EPI == EPI_DACT)
            store_block_masked<TO>(p, acc[i][j], r0, c0, lane, (w[q >> 1] >> (16 * (q & 1))) & 0xffffu);
          else
            w[q >> 1] |= store_block_bits(p, acc[i][j], r0, c0, lane) << (16 * (q & 1));
        }
      if constexpr (EPI == EPI_STORE) {
        if constexpr (MW == 4)
          *reinterpret_cast<uint4*>(mask_word) = make_uint4(w[0], w[1], w[2], w[3]);
        else
          *mask_word = w[0];
      }
    }
  } else if constexpr (EPI == EPI_DACT) {
    // The adjoint epilogue reads the saved activation (and a residual): it
    // goes through a per-wave LDS region once every wave is done with the
    // ring, so those reads and the stores move 8 consecutive columns at a time.
    static_assert(WK > 1 || NW * 32 * (WTN + 4) * 4 <= STAGES * STAGE,
                  "epilogue staging fits the ring");
    barrier_only();
    epilogue_lds<TO, EPI, TM, TN>(p, acc, reinterpret_cast<float*>(smem) + wave * 32 * (WTN + 4),
                                  m0 + wm * WTM, n0 + wn * WTN, lane);
  } else {
    // Stores only: straight from the accumulator registers, block by block.
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int i = 0; i < TM; ++i)
        store_block<bf16_t, TO, EPI>(p, acc[i][j], m0 + wm * WTM + i * 32, n0 + wn * WTN + j * 32,
                                     lane);
  }
  if constexpr (EPI == EPI_DW) {
    if (do_colsum) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const float t = cs[j] + __shfl_xor(cs[j], 32);
        const int64_t col = n0 + wn * WTN + j * 32 + lane;
        if (lane < 32 && col < p.nvec) p.colsum[col] = t;
      }
    }
  }
}

// Interleaving of matrix instructions and fragment reads per configuration
// (measured on the 256 x 256 tile with 64-deep k-tiles only).
template <int BM, int BN, int BK>
constexpr int async_ilv() { return (BM == 256 && BN == 256 && BK == 64) ? 4 : 0; }
// The k-tile barrier before the last 16-k step (buffer-descriptor loads, two
// stages), with two fragment reads per matrix instruction. Measured on the
// deep network's products on one box, alternating builds: forward 3806-3811
// against 3854-3865 us for its eight products and the output layer's, the
// seven TN+NT pairs 6180-6194 against 6314-6325, the TN product 470 against
// 480 (89.3-89.6 against 88.2-88.5 steps/s).
template <int BM, int BN, int BK, int STAGES>
constexpr bool async_early() { return BM == 256 && BN == 256 && BK == 64 && STAGES == 2; }

template <typename TO, bool AK, bool BKM, int BM, int BN, int BK, int WM, int WN, int STAGES,
          int EPI, bool PH2>
__global__ __launch_bounds__(64 * WM * WN) void dlvm_gemm_async_kernel(Params p) {
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * (BM + BN) * 2 * BK];
  constexpr int ILV = async_ilv<BM, BN, BK>();
  constexpr bool EARLY = !PH2 && async_early<BM, BN, BK, STAGES>();
  const int tile = split_slice<bf16_t, AK, BKM>(p, static_cast<int>(blockIdx.x));
  // a k-slice of a split two-phase product lies in one phase (A or A2, whose
  // extents the host passes as well: buffer-descriptor loads)
  if (PH2 && p.splits <= 1)
    async_gemm_tile<TO, AK, BKM, BM, BN, BK, WM, WN, STAGES, EPI, PH2, ILV>(p, tile, smem);
  else
    async_gemm_tile<TO, AK, BKM, BM, BN, BK, WM, WN, STAGES, EPI, false, EARLY ? 2 : ILV, true,
                    EARLY>(p, tile, smem);
}

// The same with two k-groups of WM x WN waves (WK = 2), sized for two
// workgroups per compute unit (at most 256 registers per lane).
template <typename TO, bool AK, bool BKM, int BM, int BN, int BK, int WM, int WN, int STAGES,
          int EPI, bool PH2>
__global__ __launch_bounds__(128 * WM * WN, 2) void dlvm_gemm_async_kgroup_kernel(Params p) {
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * (BM + BN) * 2 * BK];
  const int tile = split_slice<bf16_t, AK, BKM>(p, static_cast<int>(blockIdx.x));
  if (PH2 && p.splits <= 1)
    async_gemm_tile<TO, AK, BKM, BM, BN, BK, WM, WN, STAGES, EPI, PH2, 0, true, false, 2>(p, tile,
                                                                                          smem);
  else
    async_gemm_tile<TO, AK, BKM, BM, BN, BK, WM, WN, STAGES, EPI, false, 0, true, false, 2>(
        p, tile, smem);
}

// The two adjoint products of one dense layer in one launch (blocks [0, n1):
// TN wrt the weights, the rest: NT wrt the input), as dlvm_gemm_pair_kernel.
template <typename TO2, int BM, int BN, int BK, int WM, int WN, int STAGES>
__global__ __launch_bounds__(64 * WM * WN) void dlvm_gemm_async_pair_kernel(Params p1, Params p2,
                                                                            int n1) {
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * (BM + BN) * 2 * BK];
  const int b = static_cast<int>(blockIdx.x);
  constexpr bool EARLY = async_early<BM, BN, BK, STAGES>();
  constexpr int ILV = EARLY ? 2 : async_ilv<BM, BN, BK>();
  if (b < n1) {
    const int tile = split_slice<bf16_t, false, false>(p1, b);
    async_gemm_tile<float, false, false, BM, BN, BK, WM, WN, STAGES, EPI_DW, false, ILV, true,
                    EARLY>(p1, tile, smem);
  } else {
    const int tile = split_slice<bf16_t, true, true>(p2, b - n1);
    async_gemm_tile<TO2, true, true, BM, BN, BK, WM, WN, STAGES, EPI_DACT, false, ILV, true,
                    EARLY>(p2, tile, smem);
  }
}

// Configurations (bf16): BM x BN tile, k-tile depth BK, WM x WN waves, LDS ring depth.
//   10: 256 x 256, BK 64, 2 x 4 waves (128 x 64 per wave),  2 stages (128 KiB LDS)
//   11: 256 x 128, BK 64, 2 x 2 waves (128 x 64 per wave),  3 stages (144 KiB LDS)
//   12: 128 x 128, BK 64, 2 x 2 waves (64 x 64 per wave),   4 stages (128 KiB LDS)
//   13: 256 x 256, BK 32, 2 x 4 waves (128 x 64 per wave),  4 stages (128 KiB LDS)
//   16:  64 x 128, BK 64, 2 x 2 waves (32 x 64 per wave),   3 stages (72 KiB LDS: two
//        workgroups per CU); k-contiguous A only (NN, NT)
//   17: 128 x 128, BK 64, 2 x 2 waves (64 x 64 per wave),   2 stages (64 KiB LDS: two
//        workgroups per CU)
//   18:  64 x 128, BK 64, 1 x 2 waves (64 x 64 per wave) in two k-groups, 3 stages (72
//        KiB LDS: two workgroups per CU); k-contiguous A only (NN, NT)
//   19: 128 x 128, BK 64, 2 x 2 waves (64 x 64 per wave) in two k-groups, 3 stages (96
//        KiB LDS)
constexpr int kAsyncFirst = 10;

template <typename TO, bool AK, bool BKM, int EPI, bool PH2 = false>
hipError_t launch_async(const Params& p, int cfg, unsigned grid, hipStream_t s) {
  switch (cfg) {
    case 10:
      launch_kernel((dlvm_gemm_async_kernel<TO, AK, BKM, 256, 256, 64, 2, 4, 2, EPI, PH2>), dim3(grid), dim3(512), s, p);
      break;
    case 11:
      launch_kernel((dlvm_gemm_async_kernel<TO, AK, BKM, 256, 128, 64, 2, 2, 3, EPI, PH2>), dim3(grid), dim3(256), s, p);
      break;
    case 12:
      launch_kernel((dlvm_gemm_async_kernel<TO, AK, BKM, 128, 128, 64, 2, 2, 4, EPI, PH2>), dim3(grid), dim3(256), s, p);
      break;
    case 17:
      launch_kernel((dlvm_gemm_async_kernel<TO, AK, BKM, 128, 128, 64, 2, 2, 2, EPI, PH2>), dim3(grid), dim3(256), s, p);
      break;
    case 19:
      launch_kernel((dlvm_gemm_async_kgroup_kernel<TO, AK, BKM, 128, 128, 64, 2, 2, 3, EPI, PH2>), dim3(grid), dim3(512), s, p);
      break;
    case 18:
      if constexpr (AK) {
        launch_kernel((dlvm_gemm_async_kgroup_kernel<TO, AK, BKM, 64, 128, 64, 1, 2, 3, EPI, PH2>), dim3(grid), dim3(256), s, p);
        break;
      } else {
        return hipErrorInvalidValue;
      }
    case 16:
      if constexpr (AK) {  // (an m-contiguous A needs 128-row tiles)
        launch_kernel((dlvm_gemm_async_kernel<TO, AK, BKM, 64, 128, 64, 2, 2, 3, EPI, PH2>), dim3(grid), dim3(256), s, p);
        break;
      } else {
        return hipErrorInvalidValue;
      }
    default:
      launch_kernel((dlvm_gemm_async_kernel<TO, AK, BKM, 256, 256, 32, 2, 4, 4, EPI, PH2>), dim3(grid), dim3(512), s, p);
      break;
  }
  return hipGetLastError();
}

}  // namespace gemm
}  // namespace dlvm
