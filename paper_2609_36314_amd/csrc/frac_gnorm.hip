// frac_gnorm.hip -- gated RMS normalization of the layer output (gate before the
// normalization), forward and backward.  One workgroup per token row at a time;
// each thread owns up to two 8-channel vectors of the row (and the same channels in
// every row, so its weight-gradient sums need no cross-thread step).  Group sums:
// a fixed butterfly over the lanes of a group, then, for groups wider than a wave,
// the per-wave sums in order.  The weight gradient is a fixed-order sum of per-row-
// block partials, reduced by one wave per channel: repeated calls give identical bits.
#include <algorithm>

#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

constexpr int kGnNI = 2;  // 8-channel vectors per thread and row: C <= 8 * 256 * kGnNI

__device__ __forceinline__ void store8g(bf16* p, const float* v) {
  *reinterpret_cast<bf16x8*>(p) =
      bf16x8{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3], (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
}
__device__ __forceinline__ void store8g(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ float sigmg(float x) { return 1.0f / (1.0f + __expf(-x)); }

// Totals over each group of q (one value per 8-channel vector v = tid + 256 i).  NW =
// min(vectors per group, 64); wider groups add their per-wave sums (cs) in order.
// Called by every thread of the workgroup.
template <int NW>
__device__ __forceinline__ void group_totals(const float* q, float* tot, int nv, int nvg, float* cs) {
  const int tid = threadIdx.x, lane = tid & 63;
  float t[kGnNI];
#pragma unroll
  for (int i = 0; i < kGnNI; ++i) t[i] = group_allreduce<NW>(q[i], [](float x, float y) { return x + y; });
  if (nvg <= 64) {
#pragma unroll
    for (int i = 0; i < kGnNI; ++i) tot[i] = t[i];
    return;
  }
  __syncthreads();  // the previous row's readers are done with cs
#pragma unroll
  for (int i = 0; i < kGnNI; ++i) {
    const int v = tid + 256 * i;
    if (lane == 0 && v < nv) cs[v / 64] = t[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kGnNI; ++i) {
    const int v = tid + 256 * i, k0 = (v / nvg) * (nvg / 64);
    float s = 0.0f;
    if (v < nv)
      for (int k = 0; k < nvg / 64; ++k) s += cs[k0 + k];
    tot[i] = s;
  }
}

template <typename T, int NW>
__global__ void __launch_bounds__(256) frac_gnorm_fwd_kernel(GnormDims d, frac_gnorm_args a) {
  __shared__ float cs[8 * 256 * kGnNI / 8 / 64];
  const int nv = d.C / 8, nvg = d.group / 8, tid = threadIdx.x;
  for (int64_t r = blockIdx.x; r < d.rows; r += gridDim.x) {
    const T* x = reinterpret_cast<const T*>(a.x) + r * d.C;
    const T* z = reinterpret_cast<const T*>(a.z) + r * d.C;
    float u[kGnNI][8], q[kGnNI], tot[kGnNI];
#pragma unroll
    for (int i = 0; i < kGnNI; ++i) {
      const int v = tid + 256 * i;
      q[i] = 0.0f;
      if (v < nv) {
        float xv[8], zv[8];
        load8(x + v * 8, xv);
        load8(z + v * 8, zv);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          u[i][k] = xv[k] * zv[k] * sigmg(zv[k]);
          q[i] += u[i][k] * u[i][k];
        }
      }
    }
    group_totals<NW>(q, tot, nv, nvg, cs);
#pragma unroll
    for (int i = 0; i < kGnNI; ++i) {
      const int v = tid + 256 * i;
      if (v >= nv) continue;
      const float rr = rsqrtf(tot[i] / (float)d.group + a.eps);
      float y[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) y[k] = u[i][k] * rr * a.weight[v * 8 + k];
      store8g(reinterpret_cast<T*>(a.y) + r * d.C + v * 8, y);
    }
  }
}

// Rows blockIdx.x, + gridDim.x, ...; the workgroup's weight-gradient sums go to part[blockIdx.x][C].
template <typename T, int NW>
__global__ void __launch_bounds__(256) frac_gnorm_bwd_kernel(GnormDims d, frac_gnorm_bwd_args a, float* part) {
  const frac_gnorm_args& f = a.fwd;
  __shared__ float cs[8 * 256 * kGnNI / 8 / 64];
  const int nv = d.C / 8, nvg = d.group / 8, tid = threadIdx.x;
  float wacc[kGnNI][8];
#pragma unroll
  for (int i = 0; i < kGnNI; ++i)
#pragma unroll
    for (int k = 0; k < 8; ++k) wacc[i][k] = 0.0f;
  for (int64_t r = blockIdx.x; r < d.rows; r += gridDim.x) {
    const int64_t row = r * d.C;
    float xv[kGnNI][8], zv[kGnNI][8], gv[kGnNI][8], u[kGnNI][8], q[kGnNI], tot[kGnNI];
#pragma unroll
    for (int i = 0; i < kGnNI; ++i) {
      const int v = tid + 256 * i;
      q[i] = 0.0f;
      if (v < nv) {
        load8(reinterpret_cast<const T*>(f.x) + row + v * 8, xv[i]);
        load8(reinterpret_cast<const T*>(f.z) + row + v * 8, zv[i]);
        load8(reinterpret_cast<const T*>(a.dy) + row + v * 8, gv[i]);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          u[i][k] = xv[i][k] * zv[i][k] * sigmg(zv[i][k]);
          q[i] += u[i][k] * u[i][k];
        }
      }
    }
    group_totals<NW>(q, tot, nv, nvg, cs);
    float rr[kGnNI], pq[kGnNI], ptot[kGnNI];
#pragma unroll
    for (int i = 0; i < kGnNI; ++i) {
      const int v = tid + 256 * i;
      rr[i] = rsqrtf(tot[i] / (float)d.group + f.eps);
      pq[i] = 0.0f;
      if (v < nv) {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float yh = u[i][k] * rr[i];
          const float dyv = gv[i][k];
          wacc[i][k] += dyv * yh;
          gv[i][k] = dyv * f.weight[v * 8 + k];  // the gradient of yh
          pq[i] += gv[i][k] * yh;
        }
      }
    }
    group_totals<NW>(pq, ptot, nv, nvg, cs);
#pragma unroll
    for (int i = 0; i < kGnNI; ++i) {
      const int v = tid + 256 * i;
      if (v >= nv) continue;
      const float m = ptot[i] / (float)d.group;
      float dx[8], dz[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float du = rr[i] * (gv[i][k] - u[i][k] * rr[i] * m);
        const float sg = sigmg(zv[i][k]);
        dx[k] = du * zv[i][k] * sg;
        dz[k] = du * xv[i][k] * sg * (1.0f + zv[i][k] * (1.0f - sg));
      }
      store8g(reinterpret_cast<T*>(a.dx) + row + v * 8, dx);
      store8g(reinterpret_cast<T*>(a.dz) + row + v * 8, dz);
    }
  }
  if (!part) return;
#pragma unroll
  for (int i = 0; i < kGnNI; ++i) {
    const int v = tid + 256 * i;
    if (v >= nv) continue;
#pragma unroll
    for (int k = 0; k < 8; ++k) part[(int64_t)blockIdx.x * d.C + v * 8 + k] = wacc[i][k];
  }
}

// One wave per channel: lane l adds the row-block partials l, l + 64, ... in order,
// then a fixed butterfly.
__global__ void __launch_bounds__(256) frac_gnorm_reduce_kernel(GnormDims d, float* dweight, const float* part,
                                                                int nrb) {
  const int c = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (c >= d.C) return;  // wave-uniform
  float t = 0.0f;
  for (int q = lane; q < nrb; q += 64) t += part[(int64_t)q * d.C + c];
  t = group_allreduce<64>(t, [](float x, float y) { return x + y; });
  if (lane == 0) dweight[c] = t;
}

template <typename T, int NW>
hipError_t gnorm_t(const GnormDims& d, const frac_gnorm_args* fa, const frac_gnorm_bwd_args* ba, float* ws,
                   hipStream_t stream) {
  if (fa) {
    const unsigned blocks = (unsigned)std::min<int64_t>(d.rows, 8192);
    hipLaunchKernelGGL((frac_gnorm_fwd_kernel<T, NW>), dim3(blocks), dim3(256), 0, stream, d, *fa);
    return hipGetLastError();
  }
  const int nrb = (int)std::min<int64_t>(d.rows, kGnormMaxRowBlocks);
  float* part = ba->dweight ? ws : nullptr;
  hipLaunchKernelGGL((frac_gnorm_bwd_kernel<T, NW>), dim3(nrb), dim3(256), 0, stream, d, *ba, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !part) return e;
  hipLaunchKernelGGL(frac_gnorm_reduce_kernel, dim3((d.C + 3) / 4), dim3(256), 0, stream, d, ba->dweight,
                     (const float*)part, nrb);
  return hipGetLastError();
}

template <typename T>
hipError_t gnorm_k(const GnormDims& d, const frac_gnorm_args* fa, const frac_gnorm_bwd_args* ba, float* ws,
                   hipStream_t s) {
  switch (std::min(d.group / 8, 64)) {
    case 1: return gnorm_t<T, 1>(d, fa, ba, ws, s);
    case 2: return gnorm_t<T, 2>(d, fa, ba, ws, s);
    case 4: return gnorm_t<T, 4>(d, fa, ba, ws, s);
    case 8: return gnorm_t<T, 8>(d, fa, ba, ws, s);
    case 16: return gnorm_t<T, 16>(d, fa, ba, ws, s);
    case 32: return gnorm_t<T, 32>(d, fa, ba, ws, s);
    default: return gnorm_t<T, 64>(d, fa, ba, ws, s);
  }
}

}  // namespace

size_t gnorm_workspace(int64_t C) { return sizeof(float) * (size_t)kGnormMaxRowBlocks * C; }

hipError_t launch_gnorm_fwd(const GnormDims& d, const frac_gnorm_args& a, hipStream_t stream) {
  return d.bf16_io ? gnorm_k<bf16>(d, &a, nullptr, nullptr, stream) : gnorm_k<float>(d, &a, nullptr, nullptr, stream);
}

hipError_t launch_gnorm_bwd(const GnormDims& d, const frac_gnorm_bwd_args& a, float* ws, hipStream_t stream) {
  return d.bf16_io ? gnorm_k<bf16>(d, nullptr, &a, ws, stream) : gnorm_k<float>(d, nullptr, &a, ws, stream);
}

}  // namespace frac
