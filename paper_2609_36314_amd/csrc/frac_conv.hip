// frac_conv.hip -- causal depthwise 1-D convolution of the content branch
// (FracMixer, Sec. 3.3), forward and backward.  Bound by HBM: each thread owns 8
// consecutive channels (one 16-byte bfloat16 vector) of a run of 16 tokens, with its
// weights in registers and the inputs in a sliding register window (one load per
// token).  The backward recomputes the pre-activation in the window, writes dx, and
// sums the weight and bias gradients as fixed-order partials per row block, reduced
// by one wave per output: repeated calls give identical bits.
#include <algorithm>

#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

__device__ __forceinline__ void store8(bf16* p, const float* v) {
  *reinterpret_cast<bf16x8*>(p) =
      bf16x8{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3], (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
}
__device__ __forceinline__ void store8(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + __expf(-x)); }

constexpr int kConvTR = 16;  // consecutive tokens per thread

// Thread item = (b, segment of kConvTR tokens, 8-channel group), channel groups
// fastest (coalesced); the weights are loaded once and x slides through a K-token
// register window, one 16-byte load per token.
template <typename T, int K>
__global__ void __launch_bounds__(256) frac_conv_fwd_kernel(ConvDims d, frac_conv_args a) {
  const int G = d.C / 8, nseg = (d.L + kConvTR - 1) / kConvTR;
  const int64_t items = d.rows / d.L * nseg * G;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < items; i += (int64_t)gridDim.x * 256) {
    const int64_t bs = i / G;
    const int c0 = (int)(i - bs * G) * 8, b = (int)(bs / nseg), t0 = (int)(bs % nseg) * kConvTR;
    const int t1 = min(t0 + kConvTR, d.L);
    float w[8][K], bias[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      bias[q] = a.bias ? a.bias[c0 + q] : 0.0f;
#pragma unroll
      for (int j = 0; j < K; ++j) w[q][j] = a.w[(c0 + q) * K + j];
    }
    const int64_t base = (int64_t)b * d.L * d.C + c0;
    const T* x = reinterpret_cast<const T*>(a.x) + base;
    T* y = reinterpret_cast<T*>(a.y) + base;
    float xv[K][8];  // x at tokens t - (K - 1) .. t
#pragma unroll
    for (int u = 0; u < K - 1; ++u) {
      const int tt = t0 - (K - 1) + u;
      if (tt >= 0) {
        load8(x + (int64_t)tt * d.C, xv[u]);
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) xv[u][q] = 0.0f;
      }
    }
    for (int t = t0; t < t1; ++t) {
      load8(x + (int64_t)t * d.C, xv[K - 1]);
      float acc[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        float v = bias[q];
#pragma unroll
        for (int j = 0; j < K; ++j) v += w[q][j] * xv[j][q];
        acc[q] = a.activation ? v * sigm(v) : v;
      }
      store8(y + (int64_t)t * d.C, acc);
#pragma unroll
      for (int u = 0; u < K - 1; ++u)
#pragma unroll
        for (int q = 0; q < 8; ++q) xv[u][q] = xv[u + 1][q];
    }
  }
}

// Workgroup (x, y): channel groups 32 y .. 32 y + 31 (8 channels each) x 8 row lanes;
// row lane rl takes token segments (b, kConvTR tokens) 8 x + rl, then every 8 gridDim.x
// segments, each in token order with x (2K - 1 tokens) and g (K tokens) in sliding
// register windows.  Writes dx, and the workgroup's fixed-order sums of g x (weights)
// and g (bias) into pw [x][C][K], pb [x][C].
template <typename T, int K>
__global__ void __launch_bounds__(256) frac_conv_bwd_kernel(ConvDims d, frac_conv_bwd_args a, float* pw, float* pb) {
  const frac_conv_args& f = a.fwd;
  const int G = d.C / 8, nseg = (d.L + kConvTR - 1) / kConvTR;
  const int64_t segs = d.rows / d.L * nseg;
  const int cgl = threadIdx.x & 31, rl = threadIdx.x >> 5;
  const int cg = blockIdx.y * 32 + cgl, c0 = cg * 8;
  const bool active = cg < G;
  constexpr int NA = 8 * K + 8;  // accumulators per thread: weights [q][j], then bias [q]
  float acc[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) acc[i] = 0.0f;
  if (active) {
    float w[8][K], bias[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      bias[q] = f.bias ? f.bias[c0 + q] : 0.0f;
#pragma unroll
      for (int j = 0; j < K; ++j) w[q][j] = f.w[(c0 + q) * K + j];
    }
    // x at token p (zero outside the sequence); g = dL/dpre at token p (zero past the end)
    auto ldx = [&](const T* x, int p, float* o) {
      if (p >= 0 && p < d.L) {
        load8(x + (int64_t)p * d.C, o);
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] = 0.0f;
      }
    };
    for (int64_t sg = (int64_t)blockIdx.x * 8 + rl; sg < segs; sg += 8 * (int64_t)gridDim.x) {
      const int b = (int)(sg / nseg), t0 = (int)(sg % nseg) * kConvTR, t1 = min(t0 + kConvTR, d.L);
      const int64_t base = (int64_t)b * d.L * d.C + c0;
      const T* x = reinterpret_cast<const T*>(f.x) + base;
      const T* dy = reinterpret_cast<const T*>(a.dy) + base;
      T* dx = reinterpret_cast<T*>(a.dx) + base;
      float xw[2 * K - 1][8];  // x at tokens t - (K - 1) .. t + K - 1
      float g[K][8];           // g at tokens t .. t + K - 1
      auto gat = [&](int p, const float (*xs)[8], float* o) {  // xs: x at p - (K - 1) .. p
        if (p >= d.L) {
#pragma unroll
          for (int q = 0; q < 8; ++q) o[q] = 0.0f;
          return;
        }
        float gy[8];
        load8(dy + (int64_t)p * d.C, gy);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          if (f.activation) {
            float pre = bias[q];
#pragma unroll
            for (int j = 0; j < K; ++j) pre += w[q][j] * xs[j][q];
            const float sgm = sigm(pre);
            o[q] = gy[q] * (sgm + pre * sgm * (1.0f - sgm));
          } else {
            o[q] = gy[q];
          }
        }
      };
#pragma unroll
      for (int u = 0; u < 2 * K - 2; ++u) ldx(x, t0 - (K - 1) + u, xw[u]);
#pragma unroll
      for (int s = 0; s < K - 1; ++s) gat(t0 + s, xw + s, g[s]);
      for (int t = t0; t < t1; ++t) {
        ldx(x, t + K - 1, xw[2 * K - 2]);
        gat(t + K - 1, xw + (K - 1), g[K - 1]);
        float dxv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          float v = 0.0f;
#pragma unroll
          for (int j = 0; j < K; ++j) v += w[q][j] * g[K - 1 - j][q];
          dxv[q] = v;
#pragma unroll
          for (int j = 0; j < K; ++j) acc[q * K + j] += g[0][q] * xw[j][q];
          acc[8 * K + q] += g[0][q];
        }
        store8(dx + (int64_t)t * d.C, dxv);
#pragma unroll
        for (int u = 0; u < 2 * K - 2; ++u)
#pragma unroll
          for (int q = 0; q < 8; ++q) xw[u][q] = xw[u + 1][q];
#pragma unroll
        for (int s = 0; s < K - 1; ++s)
#pragma unroll
          for (int q = 0; q < 8; ++q) g[s][q] = g[s + 1][q];
      }
    }
  }
  if (!pw) return;  // workgroup-uniform
  __shared__ float red[8][32][NA + 1];
#pragma unroll
  for (int i = 0; i < NA; ++i) red[rl][cgl][i] = acc[i];
  __syncthreads();
  for (int i = threadIdx.x; i < 32 * NA; i += 256) {
    const int cl = i / NA, k = i - cl * NA, cgo = blockIdx.y * 32 + cl;
    if (cgo >= G) continue;
    float sum = 0.0f;
#pragma unroll
    for (int l = 0; l < 8; ++l) sum += red[l][cl][k];
    const int64_t base = (int64_t)blockIdx.x * d.C;
    if (k < 8 * K) {
      const int q = k / K, j = k - q * K;
      pw[(base + cgo * 8 + q) * K + j] = sum;
    } else {
      pb[base + cgo * 8 + (k - 8 * K)] = sum;
    }
  }
}

// One wave per output (C K weight gradients, then C bias gradients): lane l adds the
// row-block partials l, l + 64, ... in order, then a fixed butterfly.
__global__ void __launch_bounds__(256) frac_conv_reduce_kernel(ConvDims d, frac_conv_bwd_args a, const float* pw,
                                                               const float* pb, int nrb) {
  const int64_t o = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t nw = (int64_t)d.C * d.K;
  if (o >= nw + d.C) return;  // wave-uniform
  const bool isw = o < nw;
  if (isw ? !a.dw : !a.dbias) return;
  const float* src = isw ? pw + o : pb + (o - nw);
  const int64_t stride = isw ? nw : d.C;
  float t = 0.0f;
  for (int q = lane; q < nrb; q += 64) t += src[(int64_t)q * stride];
  t = group_allreduce<64>(t, [](float x, float y) { return x + y; });
  if (lane == 0) {
    if (isw) a.dw[o] = t;
    else a.dbias[o - nw] = t;
  }
}

template <typename T, int K>
hipError_t conv_fwd_t(const ConvDims& d, const frac_conv_args& a, hipStream_t stream) {
  const int64_t n = d.rows / d.L * ((d.L + kConvTR - 1) / kConvTR) * (d.C / 8);
  const unsigned blocks = (unsigned)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 8192));
  hipLaunchKernelGGL((frac_conv_fwd_kernel<T, K>), dim3(blocks), dim3(256), 0, stream, d, a);
  return hipGetLastError();
}

template <typename T, int K>
hipError_t conv_bwd_t(const ConvDims& d, const frac_conv_bwd_args& a, float* ws, hipStream_t stream) {
  const int64_t segs = d.rows / d.L * ((d.L + kConvTR - 1) / kConvTR);
  const int nrb = (int)std::max<int64_t>(1, std::min<int64_t>((segs + 7) / 8, kConvMaxRowBlocks));
  const bool sums = a.dw || a.dbias;
  float* pw = sums ? ws : nullptr;
  float* pb = sums ? ws + (size_t)kConvMaxRowBlocks * d.C * d.K : nullptr;
  hipLaunchKernelGGL((frac_conv_bwd_kernel<T, K>), dim3(nrb, (d.C / 8 + 31) / 32), dim3(256), 0, stream, d, a, pw,
                     pb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !sums) return e;
  const int64_t outs = (int64_t)d.C * d.K + d.C;
  hipLaunchKernelGGL(frac_conv_reduce_kernel, dim3((unsigned)((outs + 3) / 4)), dim3(256), 0, stream, d, a,
                     (const float*)pw, (const float*)pb, nrb);
  return hipGetLastError();
}

template <typename T>
hipError_t conv_fwd_k(const ConvDims& d, const frac_conv_args& a, hipStream_t s) {
  switch (d.K) {
    case 1: return conv_fwd_t<T, 1>(d, a, s);
    case 2: return conv_fwd_t<T, 2>(d, a, s);
    case 3: return conv_fwd_t<T, 3>(d, a, s);
    default: return conv_fwd_t<T, 4>(d, a, s);
  }
}

template <typename T>
hipError_t conv_bwd_k(const ConvDims& d, const frac_conv_bwd_args& a, float* ws, hipStream_t s) {
  switch (d.K) {
    case 1: return conv_bwd_t<T, 1>(d, a, ws, s);
    case 2: return conv_bwd_t<T, 2>(d, a, ws, s);
    case 3: return conv_bwd_t<T, 3>(d, a, ws, s);
    default: return conv_bwd_t<T, 4>(d, a, ws, s);
  }
}

}  // namespace

size_t conv_workspace(int64_t C, int K) { return sizeof(float) * (size_t)kConvMaxRowBlocks * C * (K + 1); }

hipError_t launch_conv_fwd(const ConvDims& d, const frac_conv_args& a, hipStream_t stream) {
  return d.bf16_io ? conv_fwd_k<bf16>(d, a, stream) : conv_fwd_k<float>(d, a, stream);
}

hipError_t launch_conv_bwd(const ConvDims& d, const frac_conv_bwd_args& a, float* ws, hipStream_t stream) {
  return d.bf16_io ? conv_bwd_k<bf16>(d, a, ws, stream) : conv_bwd_k<float>(d, a, ws, stream);
}

}  // namespace frac
