// frac_conv.hip -- causal depthwise 1-D convolution of the content branch
// (FracMixer, Sec. 3.3), forward and backward.  Bound by HBM: each thread owns 8
// consecutive channels (one 16-byte bfloat16 vector) of one token and reads the
// K - 1 earlier tokens of the same channels from cache.  The backward recomputes
// the pre-activation in a (2K - 1)-token window, writes dx, and sums the weight and
// bias gradients as fixed-order partials per row block, reduced by one wave per
// output: repeated calls give identical bits.
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

template <typename T, int K>
__global__ void __launch_bounds__(256) frac_conv_fwd_kernel(ConvDims d, frac_conv_args a) {
  const int G = d.C / 8;
  const int64_t n = d.rows * G;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t row = i / G;
    const int c0 = (int)(i - row * G) * 8, t = (int)(row % d.L);
    const T* x = reinterpret_cast<const T*>(a.x) + row * d.C + c0;
    float acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = a.bias ? a.bias[c0 + q] : 0.0f;
#pragma unroll
    for (int j = 0; j < K; ++j) {
      const int back = K - 1 - j;  // tap j reads the token `back` steps earlier
      if (t < back) continue;
      float v[8];
      load8(x - (int64_t)back * d.C, v);
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] += a.w[(c0 + q) * K + j] * v[q];
    }
    if (a.activation) {
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] *= sigm(acc[q]);
    }
    store8(reinterpret_cast<T*>(a.y) + row * d.C + c0, acc);
  }
}

// Workgroup (x, y): channel groups 32 y .. 32 y + 31 (8 channels each) x 8 row lanes;
// row lane rl takes rows 8 x + rl, then every 8 gridDim.x rows.  Writes dx, and the
// workgroup's fixed-order sums of g x (weights) and g (bias) into pw [x][C][K], pb [x][C].
template <typename T, int K>
__global__ void __launch_bounds__(256) frac_conv_bwd_kernel(ConvDims d, frac_conv_bwd_args a, float* pw, float* pb) {
  const frac_conv_args& f = a.fwd;
  const int G = d.C / 8;
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
    for (int64_t r = (int64_t)blockIdx.x * 8 + rl; r < d.rows; r += 8 * (int64_t)gridDim.x) {
      const int t = (int)(r % d.L);
      const T* x = reinterpret_cast<const T*>(f.x) + r * d.C + c0;
      const T* dy = reinterpret_cast<const T*>(a.dy) + r * d.C + c0;
      // x at tokens t - (K - 1) .. t + K - 1 of this sequence (zero outside it)
      float xw[2 * K - 1][8];
#pragma unroll
      for (int u = 0; u < 2 * K - 1; ++u) {
        const int off = u - (K - 1), tt = t + off;
        if (tt >= 0 && tt < d.L) {
          load8(x + (int64_t)off * d.C, xw[u]);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) xw[u][q] = 0.0f;
        }
      }
      // g = dL/dpre at tokens t .. t + K - 1
      float g[K][8];
#pragma unroll
      for (int s = 0; s < K; ++s) {
        if (t + s >= d.L) {
#pragma unroll
          for (int q = 0; q < 8; ++q) g[s][q] = 0.0f;
          continue;
        }
        float gy[8];
        load8(dy + (int64_t)s * d.C, gy);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          if (f.activation) {
            float pre = bias[q];
#pragma unroll
            for (int j = 0; j < K; ++j) pre += w[q][j] * xw[s + j][q];
            const float sg = sigm(pre);
            g[s][q] = gy[q] * (sg + pre * sg * (1.0f - sg));
          } else {
            g[s][q] = gy[q];
          }
        }
      }
      // dx[t] = sum_j w_j g[t + K - 1 - j]
      float dxv[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        float v = 0.0f;
#pragma unroll
        for (int j = 0; j < K; ++j) v += w[q][j] * g[K - 1 - j][q];
        dxv[q] = v;
      }
      store8(reinterpret_cast<T*>(a.dx) + r * d.C + c0, dxv);
      // dw[q][j] += g[t] x[t - (K - 1) + j], dbias[q] += g[t]
#pragma unroll
      for (int q = 0; q < 8; ++q) {
#pragma unroll
        for (int j = 0; j < K; ++j) acc[q * K + j] += g[0][q] * xw[j][q];
        acc[8 * K + q] += g[0][q];
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
    float s = 0.0f;
#pragma unroll
    for (int l = 0; l < 8; ++l) s += red[l][cl][k];
    const int64_t base = (int64_t)blockIdx.x * d.C;
    if (k < 8 * K) {
      const int q = k / K, j = k - q * K;
      pw[(base + cgo * 8 + q) * K + j] = s;
    } else {
      pb[base + cgo * 8 + (k - 8 * K)] = s;
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
  const int64_t n = d.rows * (d.C / 8);
  const unsigned blocks = (unsigned)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 8192));
  hipLaunchKernelGGL((frac_conv_fwd_kernel<T, K>), dim3(blocks), dim3(256), 0, stream, d, a);
  return hipGetLastError();
}

template <typename T, int K>
hipError_t conv_bwd_t(const ConvDims& d, const frac_conv_bwd_args& a, float* ws, hipStream_t stream) {
  const int nrb = (int)std::max<int64_t>(1, std::min<int64_t>((d.rows + 7) / 8, kConvMaxRowBlocks));
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
