// Large bf16 dense-layer products: 256 x 256 output tiles on four waves, each
// wave owning a 128 x 128 block (sixteen 32 x 32 accumulator blocks, held in
// the accumulation registers).
//
// Same products, LDS layouts, fragment reads and fused epilogues as the
// direct-to-LDS kernel of gemm_async.hpp; what changes is the balance of the
// compute unit's resources:
//
// * LDS traffic. Per 16 k a wave reads 4 A and 4 B fragments (8 KiB) for 16
//   matrix instructions, half the fragment bytes per instruction of a
//   128 x 64 wave block, so the LDS read bandwidth is no longer on a par with
//   the matrix cores.
// * Addressing. Operands are read with buffer_load ... lds through a buffer
//   descriptor: every lane's byte offset from the k-tile's first element is
//   computed once, and advancing to the next k-tile only moves the
//   descriptor's base and shrinks its size (scalar work). The hardware checks
//   each lane's offset against the descriptor's size and returns zero past it,
//   so rows past M or N need no clamping and no read leaves the operand; k
//   past K inside a row is zeroed in LDS before the last k-tile is
//   multiplied, as in the other kernels.
// * An LDS ring of STAGES k-tiles of BK k (A and B tiles of 256 x BK bf16,
//   128 KiB in all): up to STAGES - 1 k-tiles are in flight while the
//   current one is multiplied, with one barrier per k-tile; the loads of the
//   next k-tile are spread over the current one's matrix instructions, and the
//   fragments of the next 16 k are read while the matrix cores work on the
//   current ones.
#pragma once

#include "gemm_async.hpp"

namespace dlvm {
namespace gemm {

// Issue this wave's loads of one operand tile. The descriptor starts at the
// k-tile's first element: `skip` bytes into an operand of `bytes` bytes.
template <int LOADS>
__device__ __forceinline__ void xl_issue(const void* base, uint32_t bytes, uint32_t skip,
                                         const uint32_t* off, char* lds_tile, int wave) {
  const __amdgpu_buffer_rsrc_t rsrc =
      make_rsrc(static_cast<const char*>(base) + skip, bytes - skip);
#pragma unroll
  for (int j = 0; j < LOADS; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, DLVM_LDS_PTR(lds_tile + (wave * LOADS + j) * 1024), 16, off[j], 0, 0, 0);
}

// One k-tile of the wave's 4 x 4 blocks. The fragments of the next 16 k are
// read from LDS while the matrix cores work on the current ones, and this
// wave's loads of a later k-tile (if `load`) are spread over the 16 k steps
// instead of being issued in one burst.
template <bool AK, bool BKM, int BK, int LOADS, bool CS>
__device__ __forceinline__ void xl_ktile(const char* __restrict__ As, const char* __restrict__ Bs,
                                         int arow, int brow, int lane, f32x16 (&acc)[4][4],
                                         float (&cs)[4], bool do_cs, bool load,
                                         __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb,
                                         const uint32_t* offa, const uint32_t* offb,
                                         char* dst, int wave) {
  constexpr int S = BK / 16;
  constexpr int PER = LOADS / S;  // wave loads of each operand per 16 k
  static_assert(LOADS % S == 0, "loads spread evenly over the k steps");
  bf16x8 af[2][4], bfr[2][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) af[0][i] = frag<AK, 256, BK>(As, arow + i * 32, 0, lane);
#pragma unroll
  for (int j = 0; j < 4; ++j) bfr[0][j] = frag<BKM, 256, BK>(Bs, brow + j * 32, 0, lane);
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int cur = s & 1, nxt = cur ^ 1;
    if (load) {
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int j = s * PER + q;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            ra, DLVM_LDS_PTR(dst + (wave * LOADS + j) * 1024), 16, offa[j], 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rb, DLVM_LDS_PTR(dst + 256 * 2 * BK + (wave * LOADS + j) * 1024), 16, offb[j], 0, 0, 0);
      }
    }
    if (s + 1 < S) {
#pragma unroll
      for (int i = 0; i < 4; ++i) af[nxt][i] = frag<AK, 256, BK>(As, arow + i * 32, s + 1, lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) bfr[nxt][j] = frag<BKM, 256, BK>(Bs, brow + j * 32, s + 1, lane);
    }
    // Keep the reads of the next fragments ahead of this step's 16 matrix
    // instructions (the scheduler would otherwise interleave them one
    // fragment at a time and wait for each read).
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (CS) {
      if (do_cs) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
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

template <typename TO, bool AK, bool BKM, int BK, int STAGES, int EPI>
__global__ __launch_bounds__(256) void dlvm_gemm_xl_kernel(Params p) {
  constexpr int BM = 256, BN = 256;
  constexpr int WTM = 128, WTN = 128, TM = 4, TN = 4;
  constexpr int A_BYTES = BM * 2 * BK, B_BYTES = BN * 2 * BK;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int LOADS = A_BYTES / 1024 / 4;  // wave instructions per operand tile and wave
  static_assert(STAGES >= 2 && STAGES - 2 <= 3, "ring depth");
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_of(split_slice<bf16_t, AK, BKM>(p, static_cast<int>(blockIdx.x)), p.tiles_m, p.tiles_n,
          tm, tn);
  const int64_t m0 = static_cast<int64_t>(tm) * BM;
  const int64_t n0 = static_cast<int64_t>(tn) * BN;
  const int nk = static_cast<int>((p.K + BK - 1) / BK);
  const int kv_last = static_cast<int>(p.K - static_cast<int64_t>(nk - 1) * BK);

  uint32_t offa[LOADS], offb[LOADS];
  xl_offsets<AK, BK, LOADS>(offa, wave, lane, p.lda, m0);
  xl_offsets<BKM, BK, LOADS>(offb, wave, lane, p.ldb, n0);
  // Byte step of the operands' k-tile origin.
  const uint32_t stepa = AK ? BK * 2 : static_cast<uint32_t>(BK * p.lda * 2);
  const uint32_t stepb = BKM ? BK * 2 : static_cast<uint32_t>(BK * p.ldb * 2);

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  float cs[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) cs[j] = 0.0f;
  const bool do_colsum = (EPI == EPI_DW) && (p.colsum != nullptr) && (tm == 0) && (wm == 0);

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s) {
    if (s < nk) {
      char* st = smem + s * STAGE;
      xl_issue<LOADS>(p.A, p.a_bytes, static_cast<uint32_t>(s) * stepa, offa, st, wave);
      xl_issue<LOADS>(p.B, p.b_bytes, static_cast<uint32_t>(s) * stepb, offb, st + A_BYTES, wave);
    }
  }

  for (int kt = 0; kt < nk; ++kt) {
    // Stage kt has landed once at most `ahead` later stages are outstanding.
    const int left = nk - 1 - kt;
    wait_stage<2 * LOADS, STAGES - 2>(left < STAGES - 2 ? left : STAGES - 2);
    barrier_only();
    char* As = smem + (kt % STAGES) * STAGE;
    char* Bs = As + A_BYTES;
    if (kt == nk - 1 && kv_last < BK) {
      zero_k_tail<AK, BM, BK, 256>(As, kv_last, tid);
      zero_k_tail<BKM, BN, BK, 256>(Bs, kv_last, tid);
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the LDS writes are done
      barrier_only();
    }
    // The slot refilled during this k-tile was last read in iteration kt - 1,
    // before the barrier.
    const int kn = kt + STAGES - 1;
    const bool load = kn < nk;
    const uint32_t skipa = load ? static_cast<uint32_t>(kn) * stepa : 0u;
    const uint32_t skipb = load ? static_cast<uint32_t>(kn) * stepb : 0u;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(static_cast<const char*>(p.A) + skipa, p.a_bytes - skipa);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(static_cast<const char*>(p.B) + skipb, p.b_bytes - skipb);
    xl_ktile<AK, BKM, BK, LOADS, EPI == EPI_DW>(As, Bs, wm * WTM, wn * WTN, lane, acc, cs, do_colsum,
                                                load, ra, rb, offa, offb,
                                                smem + (kn % STAGES) * STAGE, wave);
  }

  // Epilogue through a per-wave LDS region once every wave is done with the ring.
  static_assert(4 * 32 * (WTN + 4) * 4 <= STAGES * STAGE, "epilogue staging fits the ring");
  barrier_only();
  epilogue_lds<TO, EPI, TM, TN>(p, acc, reinterpret_cast<float*>(smem) + wave * 32 * (WTN + 4),
                                m0 + wm * WTM, n0 + wn * WTN, lane);
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

// Configurations 14 (64-deep k-tiles, 2 stages) and 15 (32-deep k-tiles, 4
// stages) are this kernel; the other bf16 configurations from 10 on are the
// kernels of gemm_async.hpp.
template <typename TO, bool AK, bool BKM, int EPI>
hipError_t launch_bf16(const Params& p, int cfg, unsigned grid, hipStream_t s) {
  switch (cfg) {
    case 14:
      launch_kernel((dlvm_gemm_xl_kernel<TO, AK, BKM, 64, 2, EPI>), dim3(grid), dim3(256), s, p);
      return hipGetLastError();
    case 15:
      launch_kernel((dlvm_gemm_xl_kernel<TO, AK, BKM, 32, 4, EPI>), dim3(grid), dim3(256), s, p);
      return hipGetLastError();
    default:
      return launch_async<TO, AK, BKM, EPI>(p, cfg, grid, s);
  }
}

}  // namespace gemm
}  // namespace dlvm
