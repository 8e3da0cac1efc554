// frac_params.hip -- parameter construction of the control branch (FracMixer,
// Sec. 3.3): step, fractional order and scale from their projections, gated read /
// write logits, and the backward of all of it.  Elementwise and bound by HBM: one
// pass over the [B,L,H] controls and the [B,L,H,M] logits; the two reductions of
// the backward (the bias gradient per head, the two gate gradients) are fixed-order
// sums of per-block partials, so repeated calls give identical bits.
#include <algorithm>

#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

__device__ __forceinline__ float softplus_f(float x) { return x > 20.0f ? x : log1pf(expf(x)); }
__device__ __forceinline__ float sigmoid_f(float x) { return 1.0f / (1.0f + expf(-x)); }
// clip to [lo, hi]; its derivative (1 on the closed range) through *pass
__device__ __forceinline__ float clip_f(float v, float lo, float hi, float* pass) {
  *pass = (v >= lo && v <= hi) ? 1.0f : 0.0f;
  return fminf(fmaxf(v, lo), hi);
}

__global__ void __launch_bounds__(256) frac_params_fwd_kernel(ParamsDims d, frac_params_args a) {
  const int64_t nctl = d.rows * d.H, nlg = nctl * d.M;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nctl; i += stride) {
    const int h = (int)(i % d.H);
    float pass;
    a.dt[i] = clip_f(softplus_f(a.z_dt[i] + (a.dt_bias ? a.dt_bias[h] : 0.0f)), a.dt_min, a.dt_max, &pass);
    a.alpha[i] = sigmoid_f(a.z_alpha[i]);
    if (a.z_lambda) a.lambda[i] = clip_f(softplus_f(a.z_lambda[i]), a.lambda_min, a.lambda_max, &pass);
  }
  const float gr = a.v_read ? sigmoid_f(*a.p_read) : 0.0f, gw = a.v_write ? sigmoid_f(*a.p_write) : 0.0f;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nlg; i += stride) {
    if (a.v_read) a.read_logit[i] = gr * a.v_read[i];
    if (a.v_write) a.write_logit[i] = gw * a.v_write[i];
  }
}

// Elementwise gradients; per block, the fixed-order partial sums of dlogit * v for
// the two gates into part[2 block + {0, 1}].
__global__ void __launch_bounds__(256) frac_params_bwd_kernel(ParamsDims d, frac_params_bwd_args a, float* part) {
  const frac_params_args& f = a.fwd;
  const int64_t nctl = d.rows * d.H, nlg = nctl * d.M;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nctl; i += stride) {
    const int h = (int)(i % d.H);
    float pass;
    if (a.dz_dt) {
      const float x = f.z_dt[i] + (f.dt_bias ? f.dt_bias[h] : 0.0f);
      clip_f(softplus_f(x), f.dt_min, f.dt_max, &pass);
      a.dz_dt[i] = a.ddt ? a.ddt[i] * pass * sigmoid_f(x) : 0.0f;
    }
    if (a.dz_alpha) {
      const float s = sigmoid_f(f.z_alpha[i]);
      a.dz_alpha[i] = a.dalpha ? a.dalpha[i] * s * (1.0f - s) : 0.0f;
    }
    if (a.dz_lambda && f.z_lambda) {
      const float z = f.z_lambda[i];
      clip_f(softplus_f(z), f.lambda_min, f.lambda_max, &pass);
      a.dz_lambda[i] = a.dlambda ? a.dlambda[i] * pass * sigmoid_f(z) : 0.0f;
    }
  }
  const float gr = f.v_read ? sigmoid_f(*f.p_read) : 0.0f, gw = f.v_write ? sigmoid_f(*f.p_write) : 0.0f;
  float sr = 0.0f, sw = 0.0f;  // sum of dlogit * v over this thread's elements, in order
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nlg; i += stride) {
    if (f.v_read) {
      const float g = a.dread_logit ? a.dread_logit[i] : 0.0f;
      if (a.dv_read) a.dv_read[i] = gr * g;
      sr += g * f.v_read[i];
    }
    if (f.v_write) {
      const float g = a.dwrite_logit ? a.dwrite_logit[i] : 0.0f;
      if (a.dv_write) a.dv_write[i] = gw * g;
      sw += g * f.v_write[i];
    }
  }
  sr = group_allreduce<64>(sr, [](float x, float y) { return x + y; });
  sw = group_allreduce<64>(sw, [](float x, float y) { return x + y; });
  __shared__ float red[2][4];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) {
    red[0][wave] = sr;
    red[1][wave] = sw;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    const float* r = red[threadIdx.x];
    part[2 * blockIdx.x + threadIdx.x] = (r[0] + r[1]) + (r[2] + r[3]);
  }
}

// Partial bias gradients: workgroup (x, y) sums rows x*4 + lane/64 + k*4*gridDim.x
// of heads 64 y + lane%64 in order, then its 4 row lanes in order, into pb[x][h].
__global__ void __launch_bounds__(256) frac_params_bias_kernel(ParamsDims d, frac_params_bwd_args a, float* pb) {
  const frac_params_args& f = a.fwd;
  __shared__ float acc[4][64];
  const int hh = threadIdx.x & 63, rl = threadIdx.x >> 6, h = blockIdx.y * 64 + hh;
  float s = 0.0f;
  if (h < d.H && a.ddt) {
    const float b = f.dt_bias ? f.dt_bias[h] : 0.0f;
    for (int64_t r = (int64_t)blockIdx.x * 4 + rl; r < d.rows; r += 4 * (int64_t)gridDim.x) {
      const int64_t i = r * d.H + h;
      const float x = f.z_dt[i] + b;
      float pass;
      clip_f(softplus_f(x), f.dt_min, f.dt_max, &pass);
      s += a.ddt[i] * pass * sigmoid_f(x);
    }
  }
  acc[rl][hh] = s;
  __syncthreads();
  if (rl == 0 && h < d.H) pb[(int64_t)blockIdx.x * d.H + h] = (acc[0][hh] + acc[1][hh]) + (acc[2][hh] + acc[3][hh]);
}

// One wave per output: the bias gradient of each head (from the row-block partials)
// and the two gate gradients (from the per-block partials).  Lane j adds partials
// j, j + 64, ... in order, then the lanes are combined by a fixed butterfly.
__global__ void __launch_bounds__(256) frac_params_reduce_kernel(ParamsDims d, frac_params_bwd_args a,
                                                                 const float* part, int nblocks, const float* pb,
                                                                 int nrb) {
  const frac_params_args& f = a.fwd;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;  // wave-uniform output
  auto wave_sum = [&](const float* src, int n, int64_t stride) {
    float t = 0.0f;
    for (int q = lane; q < n; q += 64) t += src[(int64_t)q * stride];
    return group_allreduce<64>(t, [](float x, float y) { return x + y; });
  };
  if (o < d.H) {
    if (!a.ddt_bias) return;
    const float t = wave_sum(pb + o, nrb, d.H);
    if (lane == 0) a.ddt_bias[o] = t;
  } else if (o < d.H + 2) {
    const bool rd = o == d.H;
    float* out = rd ? a.dp_read : a.dp_write;
    if (!out) return;
    if (!(rd ? f.v_read : f.v_write)) {
      if (lane == 0) *out = 0.0f;
      return;
    }
    const float t = wave_sum(part + (rd ? 0 : 1), nblocks, 2);
    const float g = sigmoid_f(*(rd ? f.p_read : f.p_write));
    if (lane == 0) *out = t * g * (1.0f - g);
  }
}

}  // namespace

hipError_t launch_params_fwd(const ParamsDims& d, const frac_params_args& a, hipStream_t stream) {
  const int64_t n = d.rows * d.H * (a.v_read || a.v_write ? d.M : 1);
  const unsigned blocks = (unsigned)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 4096));
  hipLaunchKernelGGL(frac_params_fwd_kernel, dim3(blocks), dim3(256), 0, stream, d, a);
  return hipGetLastError();
}

size_t params_workspace(int64_t H) { return sizeof(float) * (2 * kParamsMaxBlocks + (size_t)kParamsMaxBlocks * H); }

hipError_t launch_params_bwd(const ParamsDims& d, const frac_params_bwd_args& a, float* part, hipStream_t stream) {
  const int64_t n = d.rows * d.H * d.M;
  const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, kParamsMaxBlocks));
  hipLaunchKernelGGL(frac_params_bwd_kernel, dim3(blocks), dim3(256), 0, stream, d, a, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  float* pb = part + 2 * kParamsMaxBlocks;  // [nrb][H]
  const int nrb = (int)std::max<int64_t>(1, std::min<int64_t>((d.rows + 3) / 4, kParamsMaxBlocks));
  if (a.ddt_bias) {
    hipLaunchKernelGGL(frac_params_bias_kernel, dim3(nrb, (d.H + 63) / 64), dim3(256), 0, stream, d, a, pb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(frac_params_reduce_kernel, dim3((d.H + 2 + 3) / 4), dim3(256), 0, stream, d, a,
                     (const float*)part, blocks, (const float*)pb, nrb);
  return hipGetLastError();
}

}  // namespace frac
