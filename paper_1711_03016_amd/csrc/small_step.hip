// The whole gradient of a small float32 softmax network in one workgroup.
//
// When the input, every weight and every layer output of a network fit in one
// compute unit's LDS and the products are tiny (the 64-32-10 network at batch
// 16 does 81K multiply-adds a step), a launch costs more than the work: the
// usual plan's launches are host-bound. Here one workgroup of 1024 threads
//   stages    the parameter block (every W_l and b_l, as it lies in memory),
//             x and the labels into LDS with plain contiguous copies (16-byte
//             loads where whole), all loads issued before the first store so
//             that HBM latency is paid once;
//   forward   H_{l+1} = act_l(H_l . W_l + b_l), the last layer giving logits;
//   loss      softmax cross-entropy, one wave per row, and the adjoint of the
//             logits (p - onehot) / B;
//   adjoint   per layer from the last: dW_l = H_l^T dZ, db_l = colsum dZ,
//             dZ_{l-1} = (dZ . W_l^T) * act'(H_l) (dx = dZ . W_0^T when x is
//             differentiated; the first layer's input adjoint is otherwise dead);
//   finalise  the mean loss, the device flags, the padding of dparams zeroed;
// with workgroup barriers between the phases and nothing but the results
// written to global memory. A phase with fewer outputs than threads gives each
// output a group of T adjacent lanes (T the largest power of two, at most 16,
// with T x outputs <= 1024): lane q of the group sums the terms q, q + T, ...
// and a butterfly over the group adds the T partial sums. Every sum thus runs
// in a fixed order, so the result is the same on every run. Products are
// plain float32 fused multiply-adds: at these sizes the matrix cores would
// not be fed.
//
// LDS layout (words): the parameter block (W_l as [w_l][ldw_l], b_l, the
// padding between them); H_0 .. H_L as [B][w_l]; two adjoint buffers
// [B][maxw]; row losses, row label marks and labels [B] each.
#include "common.hpp"
#include "kernels.hpp"

namespace dlvm {
namespace {

constexpr int kWaves = kSmallThreads / 64;
constexpr int kStage4 = kSmallMaxLds / 16 / kSmallThreads;  // 16-byte loads per thread and block

__device__ __forceinline__ float wave_sum(float v) {
  // butterfly: every lane ends with the same bits
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ int wave_or(int v) {
  for (int o = 32; o > 0; o >>= 1) v |= __shfl_xor(v, o);
  return v;
}

// Lanes per output for a phase of `outputs` sums (uniform over the workgroup).
__device__ __forceinline__ int group_lanes(int outputs) {
  int t = 1;
  while (t < 16 && 2 * t * outputs <= kSmallThreads) t *= 2;
  return t;
}

// Sum of v over the T adjacent lanes of a group (T a power of two <= 16;
// every lane of the group active).
__device__ __forceinline__ float group_sum(float v, int T) {
  for (int o = T >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__global__ __launch_bounds__(kSmallThreads) void dlvm_small_step_kernel(
    SmallNet t, const float* __restrict__ params, const float* __restrict__ x,
    const int32_t* __restrict__ labels, float* __restrict__ loss, float* __restrict__ dparams,
    float* __restrict__ dx, int32_t* __restrict__ flags, ZeroGaps gaps) {
  __shared__ __attribute__((aligned(16))) float sm[kSmallMaxLds / 4];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int B = t.B;

  // stage the parameter block, x and the labels (16-byte body, word tail)
  {
    const float* pb = params + t.pbase;
    const int np4 = t.pwords / 4, nx = B * t.w[0], nx4 = nx / 4;
    float4 pv[kStage4], xv[kStage4];
#pragma unroll
    for (int j = 0; j < kStage4; ++j) {
      const int e = tid + j * kSmallThreads;
      if (e < np4) pv[j] = reinterpret_cast<const float4*>(pb)[e];
      if (e < nx4) xv[j] = reinterpret_cast<const float4*>(x)[e];
    }
    const int pt = np4 * 4 + tid, xt = nx4 * 4 + tid;
    const float ptail = pt < t.pwords ? pb[pt] : 0.0f;
    const float xtail = xt < nx ? x[xt] : 0.0f;
    const int lab = tid < B ? labels[tid] : 0;
    float* xs = sm + t.hoff[0];
#pragma unroll
    for (int j = 0; j < kStage4; ++j) {
      const int e = tid + j * kSmallThreads;
      if (e < np4) reinterpret_cast<float4*>(sm)[e] = pv[j];
      if (e < nx4) reinterpret_cast<float4*>(xs)[e] = xv[j];
    }
    if (pt < t.pwords) sm[pt] = ptail;
    if (xt < nx) xs[xt] = xtail;
    if (tid < B) reinterpret_cast<int*>(sm + t.labels)[tid] = lab;
  }
  __syncthreads();

  // forward
  for (int l = 0; l < t.L; ++l) {
    const int K = t.w[l], N = t.w[l + 1], sw = t.ldw[l], act = t.act[l];
    const float* h = sm + t.hoff[l];
    const float* W = sm + t.woff[l];
    const float* bias = sm + t.boff[l];
    float* o = sm + t.hoff[l + 1];
    const bool last = l == t.L - 1;
    const int T = group_lanes(B * N), q = tid & (T - 1);
    for (int i = tid / T; i < B * N; i += kSmallThreads / T) {
      const int r = i / N, n = i - r * N;
      const float* hr = h + r * K;
      float acc = 0.0f;
#pragma unroll 4
      for (int k = q; k < K; k += T) acc = fmaf(hr[k], W[k * sw + n], acc);
      acc = group_sum(acc, T) + bias[n];
      if (q == 0) o[i] = last ? acc : apply_act(act, acc);
    }
    __syncthreads();
  }

  // softmax cross-entropy, one wave per row; the adjoint of the logits
  const int C = t.w[t.L];
  const float* Z = sm + t.hoff[t.L];
  float* rowloss = sm + t.rowloss;
  int* rowbad = reinterpret_cast<int*>(sm + t.rowbad);
  const int* lab = reinterpret_cast<const int*>(sm + t.labels);
  float* g = sm + t.g0;
  float* gn = sm + t.g1;
  for (int r = wave; r < B; r += kWaves) {
    const float* z = Z + r * C;
    float m = -INFINITY;
    for (int c = lane; c < C; c += 64) m = fmaxf(m, z[c]);
    m = wave_max(m);
    float s = 0.0f;
    for (int c = lane; c < C; c += 64) s += __expf(z[c] - m);
    s = wave_sum(s);
    const int y = lab[r];
    const bool ok = y >= 0 && y < C;
    if (lane == 0) {
      rowbad[r] = ok ? 0 : 1;
      rowloss[r] = ok ? (m + __logf(s)) - z[y] : NAN;
    }
    const float ps = t.scale / s;
    for (int c = lane; c < C; c += 64)
      g[r * C + c] = ps * __expf(z[c] - m) - (c == y ? t.scale : 0.0f);
  }
  __syncthreads();

  // the mean loss and the flags (wave 0; nothing below reads what it writes)
  if (wave == 0) {
    float s = 0.0f;
    int bad = 0;
    for (int r = lane; r < B; r += 64) {
      s += rowloss[r];
      bad |= rowbad[r];
    }
    s = wave_sum(s);
    bad = wave_or(bad);
    if (lane == 0) {
      const float lv = s * t.scale;
      loss[0] = lv;
      flags[0] = bad ? 1 : 0;
      flags[1] = isfinite(lv) ? 0 : 1;
    }
  }

  // adjoint, last layer first
  for (int l = t.L - 1; l >= 0; --l) {
    const int K = t.w[l], N = t.w[l + 1], ld = t.ldw[l];
    const float* W = sm + t.woff[l];
    const float* h = sm + t.hoff[l];
    float* dW = dparams + t.offW[l];
    float* db = dparams + t.offB[l];
    // dW [K, ld] (padding columns zero) and db [N]
    {
      const int T = group_lanes(K * ld), q = tid & (T - 1);
      for (int i = tid / T; i < K * ld; i += kSmallThreads / T) {
        const int k = i / ld, n = i - k * ld;
        float acc = 0.0f;
        if (n < N) {
#pragma unroll 4
          for (int r = q; r < B; r += T) acc = fmaf(h[r * K + k], g[r * N + n], acc);
        }
        acc = group_sum(acc, T);
        if (q == 0) dW[i] = acc;
      }
    }
    {
      const int T = group_lanes(N), q = tid & (T - 1);
      for (int n = tid / T; n < N; n += kSmallThreads / T) {
        float acc = 0.0f;
        for (int r = q; r < B; r += T) acc += g[r * N + n];
        acc = group_sum(acc, T);
        if (q == 0) db[n] = acc;
      }
    }
    if (l > 0 || t.wrt_x) {
      const int T = group_lanes(B * K), q = tid & (T - 1);
      for (int i = tid / T; i < B * K; i += kSmallThreads / T) {
        const int r = i / K, k = i - r * K;
        const float* gr = g + r * N;
        const float* wr = W + k * ld;
        float acc = 0.0f;
#pragma unroll 4
        for (int n = q; n < N; n += T) acc = fmaf(gr[n], wr[n], acc);
        acc = group_sum(acc, T);
        if (q == 0) {
          if (l > 0)
            gn[i] = acc * act_grad_from_output(t.act[l - 1], h[i]);
          else
            dx[i] = acc;
        }
      }
    }
    __syncthreads();
    float* tmp = g;
    g = gn;
    gn = tmp;
  }

  for (int q = 0; q < gaps.n; ++q)
    for (int i = tid; i < gaps.len[q]; i += kSmallThreads) dparams[gaps.off[q] + i] = 0.0f;
}

}  // namespace

bool small_net(int L, const int32_t* widths, const int32_t* acts, const int64_t* offsets,
               const int64_t* ldw, int64_t B, bool wrt_x, SmallNet& t) {
  if (L < 1 || L > kSmallMaxLayers || B < 1 || B > 1024) return false;
  t = SmallNet{};
  t.L = L;
  t.B = static_cast<int>(B);
  t.wrt_x = wrt_x ? 1 : 0;
  for (int l = 0; l <= L; ++l) {
    if (widths[l] < 1 || widths[l] > 4096) return false;
    t.w[l] = widths[l];
    t.maxw = widths[l] > t.maxw ? widths[l] : t.maxw;
  }
  // LDS layout, in words, checked against the budget before any narrowing;
  // blocks start on 4-word (16-byte) boundaries
  const int64_t pbase = offsets[0];
  const int64_t pwords = offsets[2 * L - 1] + widths[L] - pbase;
  int64_t words = 0;
  auto take = [&](int64_t n) {
    const int64_t o = words;
    words += (n + 3) / 4 * 4;
    return o;
  };
  take(pwords);
  int64_t hoff[kSmallMaxLayers + 1];
  for (int l = 0; l <= L; ++l) hoff[l] = take(B * widths[l]);
  const int64_t g0 = take(B * t.maxw), g1 = take(B * t.maxw);
  const int64_t rl = take(B), rb = take(B), lb = take(B);
  int64_t macs = 0;
  for (int l = 0; l < L; ++l) {
    if (ldw[l] > 4096) return false;
    macs += 3 * B * int64_t(widths[l]) * widths[l + 1];
  }
  if (words > kSmallMaxLds / 4 || macs > kSmallMaxMacs) return false;
  t.pbase = pbase;
  t.pwords = static_cast<int>(pwords);
  for (int l = 0; l <= L; ++l) t.hoff[l] = static_cast<int>(hoff[l]);
  t.g0 = static_cast<int>(g0);
  t.g1 = static_cast<int>(g1);
  t.rowloss = static_cast<int>(rl);
  t.rowbad = static_cast<int>(rb);
  t.labels = static_cast<int>(lb);
  for (int l = 0; l < L; ++l) {
    t.act[l] = acts[l];
    t.woff[l] = static_cast<int>(offsets[2 * l] - pbase);
    t.boff[l] = static_cast<int>(offsets[2 * l + 1] - pbase);
    t.offW[l] = offsets[2 * l];
    t.offB[l] = offsets[2 * l + 1];
    t.ldw[l] = static_cast<int>(ldw[l]);
  }
  t.scale = static_cast<float>(1.0 / static_cast<double>(B));
  return true;
}

hipError_t launch_small_step(const SmallNet& t, const float* params, const float* x,
                             const int32_t* labels, float* loss, float* dparams, float* dx,
                             int32_t* flags, const ZeroGaps& gaps, hipStream_t s) {
  if (t.pwords > kSmallMaxLds / 4 || t.B * t.w[0] > kSmallMaxLds / 4) return hipErrorInvalidValue;
  launch_kernel(dlvm_small_step_kernel, dim3(1), dim3(kSmallThreads), s, t, params, x, labels,
                loss, dparams, dx, flags, gaps);
  return hipGetLastError();
}

}  // namespace dlvm
