// frac_decode.hip -- bounded-state decode: one token of the recurrence on a
// cached state, updated in place (the one-step recurrent form named in the remark
// closing Sec. 3.2; steps of the Appendix-D algorithm with the B/C-widened state).
//
// Per (batch, head) the step reads and rewrites the whole M x N x P float32 state
// once; everything else is a few hundred bytes.  The kernel is therefore a
// streaming kernel: one workgroup of 1024 threads per (batch, head), the state
// walked as rows of P floats with 16-byte loads and stores, the readout reduced
// over (m, n) in registers and then across row groups through LDS in a fixed
// order.  With 1024 threads a 4-mode state (128 KB) is read in one batch of
// loads and then written back, which keeps the DRAM traffic in long runs.
#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

constexpr int kDecodeThreads = 1024;
constexpr int kDecodeUnroll = 8;

// NT threads per (b, h): 1024 for large states (one batch of loads, then the writes:
// long DRAM runs), 256 when the state is at most 2048 float4 (the form without B/C),
// where more resident workgroups hide the per-token coefficient latency.
template <typename T, int MP, int NT>
__global__ void __launch_bounds__(NT) frac_decode_kernel(ScanParams p, float* __restrict__ state) {
  const int tid = threadIdx.x;
  const int H = p.H, P = p.P, N = p.N, M = p.M;
  const int bh = blockIdx.x;
  const int b = bh / H, h = bh - b * H, g = h * p.G / H;

  __shared__ float sB[128], sC[128], sx[256];
  __shared__ float s_rho[MP], s_kap[MP], s_c[MP];
  __shared__ float4 red[NT];

  const T* x = reinterpret_cast<const T*>(p.x) + ((int64_t)b * H + h) * P;
  const T* Bg = reinterpret_cast<const T*>(p.Bm) + ((int64_t)b * p.G + g) * N;
  const T* Cg = reinterpret_cast<const T*>(p.Cm) + ((int64_t)b * p.G + g) * N;

  if (tid < 64) {
    // per-token coefficients (eq. tau-eff, eq. rho-beta-def-frac, Algorithm steps 1-6):
    // lane m < MP handles mode m, the softmax runs across those lanes
    const int m = tid < MP ? tid : MP - 1;
    const int64_t ith = (int64_t)b * H + h;
    const float dtv = p.dt[ith];
    const float al = p.alpha[b * p.as0 + h * p.as1];
    const float lam = p.lambda ? p.lambda[b * p.ls0 + h * p.ls1] : 1.0f;
    const float dtt = effective_step(dtv, al, p.lambda, lam);
    const float tau = (m < M) ? p.tau[m] : 1.0f;
    const float prior = -al * logf(tau);
    const float zc = (m < M) ? prior + (p.read_logit ? p.read_logit[ith * M + m] : 0.0f) : -INFINITY;
    const float zw = (m < M) ? prior + (p.write_logit ? p.write_logit[ith * M + m] : 0.0f) : -INFINITY;
    const float cw = group_softmax<MP>(zc);
    const float ww = group_softmax<MP>(zw);
    if (tid < MP) {
      const float arg = (m < M) ? -dtt / tau : 0.0f;
      s_rho[m] = expf(arg);
      s_kap[m] = -expm1f(arg) * ww;
      s_c[m] = cw;
    }
  }
  for (int i = tid; i < N; i += NT) {  // without B/C (dstate 1) both are 1
    sB[i] = p.Bm ? to_f32(Bg[i]) : 1.0f;
    sC[i] = p.Cm ? to_f32(Cg[i]) : 1.0f;
  }
  for (int i = tid; i < P; i += NT) sx[i] = to_f32(x[i]);
  __syncthreads();

  const int P4 = P >> 2;             // float4 columns per state row
  const int RG = NT / P4;  // row groups
  const int col = tid % P4, rg = tid / P4;
  const float4 xv = make_float4(sx[4 * col], sx[4 * col + 1], sx[4 * col + 2], sx[4 * col + 3]);
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  float* base = state + ((int64_t)b * H + h) * (int64_t)M * N * P + 4 * col;

  // rows rg, rg + RG, ... of the (m, n) row space; (m, n) of a row kept incrementally
  const int rows = (rg < RG) ? M * N : 0;  // threads beyond the last full row group idle
  int m0 = 0, n0 = rg;
  while (n0 >= N) {
    n0 -= N;
    ++m0;
  }
  for (int r0 = rg; r0 < rows; r0 += RG * kDecodeUnroll) {
    // the state is touched once per step: stream it past the caches
    floatx4 s[kDecodeUnroll];
#pragma unroll
    for (int u = 0; u < kDecodeUnroll; ++u) {
      const int row = r0 + u * RG;
      if (row < rows) s[u] = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(base + (int64_t)row * P));
    }
#pragma unroll
    for (int u = 0; u < kDecodeUnroll; ++u) {
      const int row = r0 + u * RG;
      if (row < rows) {
        const float rho = s_rho[m0];
        const float kb = s_kap[m0] * sB[n0];
        floatx4 v = s[u];
        v[0] = rho * v[0] + kb * xv.x;
        v[1] = rho * v[1] + kb * xv.y;
        v[2] = rho * v[2] + kb * xv.z;
        v[3] = rho * v[3] + kb * xv.w;
        __builtin_nontemporal_store(v, reinterpret_cast<floatx4*>(base + (int64_t)row * P));
        const float cc = s_c[m0] * sC[n0];
        acc[0] += cc * v[0];
        acc[1] += cc * v[1];
        acc[2] += cc * v[2];
        acc[3] += cc * v[3];
      }
      n0 += RG;
      while (n0 >= N) {
        n0 -= N;
        ++m0;
      }
    }
  }
  red[tid] = make_float4(acc[0], acc[1], acc[2], acc[3]);
  __syncthreads();
  if (tid < P4) {
    float4 sum = red[tid];
    for (int j = 1; j < RG; ++j) {
      const float4 o = red[j * P4 + tid];
      sum.x += o.x;
      sum.y += o.y;
      sum.z += o.z;
      sum.w += o.w;
    }
    const float Dh = p.D ? p.D[h] : 0.0f;
    T* y = reinterpret_cast<T*>(p.y) + ((int64_t)b * H + h) * P + 4 * tid;
    y[0] = (T)(sum.x + Dh * sx[4 * tid]);
    y[1] = (T)(sum.y + Dh * sx[4 * tid + 1]);
    y[2] = (T)(sum.z + Dh * sx[4 * tid + 2]);
    y[3] = (T)(sum.w + Dh * sx[4 * tid + 3]);
  }
}

template <typename T, int MP>
hipError_t launch_decode_variant(const ScanParams& p, float* state, hipStream_t stream) {
  if ((int64_t)p.M * p.N * p.P / 4 <= 2048)
    hipLaunchKernelGGL((frac_decode_kernel<T, MP, 256>), dim3(p.Bsz * p.H), dim3(256), 0, stream, p, state);
  else
    hipLaunchKernelGGL((frac_decode_kernel<T, MP, kDecodeThreads>), dim3(p.Bsz * p.H), dim3(kDecodeThreads), 0,
                       stream, p, state);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_decode_mp(const ScanParams& p, float* state, hipStream_t stream) {
  if (p.M <= 1) return launch_decode_variant<T, 1>(p, state, stream);
  if (p.M <= 2) return launch_decode_variant<T, 2>(p, state, stream);
  if (p.M <= 4) return launch_decode_variant<T, 4>(p, state, stream);
  if (p.M <= 8) return launch_decode_variant<T, 8>(p, state, stream);
  if (p.M <= 16) return launch_decode_variant<T, 16>(p, state, stream);
  return launch_decode_variant<T, 32>(p, state, stream);
}

}  // namespace

hipError_t launch_decode_step(const ScanParams& p, float* state, hipStream_t stream) {
  if (p.Bsz == 0) return hipSuccess;
  return p.io_bf16 ? launch_decode_mp<bf16>(p, state, stream) : launch_decode_mp<float>(p, state, stream);
}

}  // namespace frac
