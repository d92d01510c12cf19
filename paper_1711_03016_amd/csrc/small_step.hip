// The whole gradient of a small float32 softmax network in one workgroup.
//
// When the input, every weight and every layer output of a network fit in one
// compute unit's LDS and the products are tiny (the 64-32-10 network at batch
// 16 does 81K multiply-adds a step), a launch costs more than the work: the
// usual plan's launches are host-bound. Here one workgroup of 1024 threads
//   stages    x, the labels, every W_l and b_l into LDS, all loads issued
//             before the first store so that HBM latency is paid once;
//   forward   H_{l+1} = act_l(H_l . W_l + b_l), the last layer giving logits;
//   loss      softmax cross-entropy, one wave per row, and the adjoint of the
//             logits (p - onehot) / B;
//   adjoint   per layer from the last: dW_l = H_l^T dZ, db_l = colsum dZ,
//             dZ_{l-1} = (dZ . W_l^T) * act'(H_l) (dx = dZ . W_0^T when x is
//             differentiated; the first layer's input adjoint is otherwise dead);
//   finalise  the mean loss, the device flags, the padding of dparams zeroed;
// with workgroup barriers between the phases and nothing but the results
// written to global memory. Every sum runs in a fixed order (one thread per
// output with k in order, or a fixed butterfly across a wave), so the result
// is the same on every run. Products are plain float32 fused multiply-adds:
// at these sizes the matrix cores would not be fed.
//
// LDS layout (words): H_0 .. H_L as [B][w_l]; two adjoint buffers [B][maxw];
// row losses, row label marks and labels [B] each; W_l as [w_l][sw_l] with an
// odd row stride sw_l >= w_{l+1} (the transposed read of the input adjoint
// walks down a column: an odd stride keeps its lanes on distinct banks); b_l.
#include "common.hpp"
#include "kernels.hpp"

namespace dlvm {
namespace {

constexpr int kWaves = kSmallThreads / 64;

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

__global__ __launch_bounds__(kSmallThreads) void dlvm_small_step_kernel(
    SmallNet t, const float* __restrict__ params, const float* __restrict__ x,
    const int32_t* __restrict__ labels, float* __restrict__ loss, float* __restrict__ dparams,
    float* __restrict__ dx, int32_t* __restrict__ flags, ZeroGaps gaps) {
  __shared__ float sm[kSmallMaxLds / 4];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int B = t.B;

  // stage x, labels, weights and biases
  {
    uint32_t v[kSmallStageRegs];
    int dst[kSmallStageRegs];
#pragma unroll
    for (int j = 0; j < kSmallStageRegs; ++j) {
      const int e = tid + j * kSmallThreads;
      dst[j] = -1;
      v[j] = 0;
      if (e < t.nstage) {
        int s = 0;
        while (s + 1 < t.nseg && t.seg[s + 1].start <= e) ++s;
        const SmallSeg& g = t.seg[s];
        const int q = e - g.start;
        const int r = q / g.cols, c = q - r * g.cols;
        const uint32_t* src = g.src == 0   ? reinterpret_cast<const uint32_t*>(x)
                              : g.src == 1 ? reinterpret_cast<const uint32_t*>(params)
                                           : reinterpret_cast<const uint32_t*>(labels);
        v[j] = src[g.goff + static_cast<int64_t>(r) * g.gstride + c];
        dst[j] = g.lds + r * g.lstride + c;
      }
    }
    uint32_t* smu = reinterpret_cast<uint32_t*>(sm);
#pragma unroll
    for (int j = 0; j < kSmallStageRegs; ++j)
      if (dst[j] >= 0) smu[dst[j]] = v[j];
  }
  __syncthreads();

  // forward
  for (int l = 0; l < t.L; ++l) {
    const int K = t.w[l], N = t.w[l + 1], sw = t.sw[l], act = t.act[l];
    const float* h = sm + t.hoff[l];
    const float* W = sm + t.woff[l];
    const float* bias = sm + t.boff[l];
    float* o = sm + t.hoff[l + 1];
    const bool last = l == t.L - 1;
    for (int i = tid; i < B * N; i += kSmallThreads) {
      const int r = i / N, n = i - r * N;
      const float* hr = h + r * K;
      float acc = bias[n];
      for (int k = 0; k < K; ++k) acc = fmaf(hr[k], W[k * sw + n], acc);
      o[i] = last ? acc : apply_act(act, acc);
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
    const int K = t.w[l], N = t.w[l + 1], sw = t.sw[l];
    const int ld = static_cast<int>(t.ldw[l]);
    const float* W = sm + t.woff[l];
    const float* h = sm + t.hoff[l];
    float* dW = dparams + t.offW[l];
    float* db = dparams + t.offB[l];
    // dW [K, ld] (padding columns zero) and db [N]
    for (int i = tid; i < K * ld; i += kSmallThreads) {
      const int k = i / ld, n = i - k * ld;
      float acc = 0.0f;
      if (n < N)
        for (int r = 0; r < B; ++r) acc = fmaf(h[r * K + k], g[r * N + n], acc);
      dW[i] = acc;
    }
    for (int n = tid; n < N; n += kSmallThreads) {
      float acc = 0.0f;
      for (int r = 0; r < B; ++r) acc += g[r * N + n];
      db[n] = acc;
    }
    if (l > 0 || t.wrt_x) {
      for (int i = tid; i < B * K; i += kSmallThreads) {
        const int r = i / K, k = i - r * K;
        const float* gr = g + r * N;
        const float* wr = W + k * sw;
        float acc = 0.0f;
        for (int n = 0; n < N; ++n) acc = fmaf(gr[n], wr[n], acc);
        if (l > 0)
          gn[i] = acc * act_grad_from_output(t.act[l - 1], h[i]);
        else
          dx[i] = acc;
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
  // LDS layout, in words, checked against the budget before any narrowing
  int64_t words = 0;
  auto take = [&](int64_t n) {
    const int64_t o = words;
    words += n;
    return o;
  };
  int64_t hoff[kSmallMaxLayers + 1], woff[kSmallMaxLayers], boff[kSmallMaxLayers];
  for (int l = 0; l <= L; ++l) hoff[l] = take(B * widths[l]);
  const int64_t g0 = take(B * t.maxw), g1 = take(B * t.maxw);
  const int64_t rl = take(B), rb = take(B), lb = take(B);
  int64_t macs = 0;
  for (int l = 0; l < L; ++l) {
    t.sw[l] = widths[l + 1] | 1;
    woff[l] = take(int64_t(widths[l]) * t.sw[l]);
    boff[l] = take(widths[l + 1]);
    macs += 3 * B * int64_t(widths[l]) * widths[l + 1];
  }
  if (words > kSmallMaxLds / 4 || macs > kSmallMaxMacs) return false;
  for (int l = 0; l <= L; ++l) t.hoff[l] = static_cast<int>(hoff[l]);
  t.g0 = static_cast<int>(g0);
  t.g1 = static_cast<int>(g1);
  t.rowloss = static_cast<int>(rl);
  t.rowbad = static_cast<int>(rb);
  t.labels = static_cast<int>(lb);
  for (int l = 0; l < L; ++l) {
    t.act[l] = acts[l];
    t.woff[l] = static_cast<int>(woff[l]);
    t.boff[l] = static_cast<int>(boff[l]);
    t.offW[l] = offsets[2 * l];
    t.offB[l] = offsets[2 * l + 1];
    t.ldw[l] = ldw[l];
  }
  // what the staging copies: x [B][w_0], the labels, then W_l and b_l per layer
  int start = 0;
  auto seg = [&](int src, int64_t goff, int rows, int cols, int gstride, int lds, int lstride) {
    SmallSeg& s = t.seg[t.nseg++];
    s = SmallSeg{goff, gstride, cols, lds, lstride, start, src};
    start += rows * cols;
  };
  seg(0, 0, t.B, widths[0], widths[0], t.hoff[0], widths[0]);
  seg(2, 0, 1, t.B, t.B, t.labels, t.B);
  for (int l = 0; l < L; ++l) {
    seg(1, offsets[2 * l], widths[l], widths[l + 1], static_cast<int>(ldw[l]), t.woff[l], t.sw[l]);
    seg(1, offsets[2 * l + 1], 1, widths[l + 1], widths[l + 1], t.boff[l], widths[l + 1]);
  }
  t.nstage = start;  // <= words <= kSmallThreads * kSmallStageRegs
  t.scale = static_cast<float>(1.0 / static_cast<double>(B));
  return true;
}

hipError_t launch_small_step(const SmallNet& t, const float* params, const float* x,
                             const int32_t* labels, float* loss, float* dparams, float* dx,
                             int32_t* flags, const ZeroGaps& gaps, hipStream_t s) {
  if (t.nstage > kSmallThreads * kSmallStageRegs) return hipErrorInvalidValue;
  launch_kernel(dlvm_small_step_kernel, dim3(1), dim3(kSmallThreads), s, t, params, x, labels,
                loss, dparams, dx, flags, gaps);
  return hipGetLastError();
}

}  // namespace dlvm
