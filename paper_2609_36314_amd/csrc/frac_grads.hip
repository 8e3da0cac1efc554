// frac_grads.hip -- gradients of the step sizes, the fractional orders, lambda and
// the read / write logits, from the per-(token, mode) partials that the reverse
// sweeps of both scan forms produce:
//
//   dc_{t,m} = dL/dc_{t,m} = <C_t^T S_{t,m}, dy_t>       (the read weight, eq. frac-readout)
//   dk_{t,m} = dL/dkappa_{t,m} = <B_t^T dS_{t,m}, x_t>   (the write gain kappa = beta w,
//                                                         eq. frac-selective-update)
//
// with S_{t,m} the state after token t and dS_{t,m} its adjoint.  Everything else is
// the chain rule through the per-token coefficients of the Appendix-D algorithm:
//
//   c = softmax_m(-alpha ln tau_m + read_logit),  w = softmax_m(-alpha ln tau_m + write_logit)
//   beta_m = 1 - rho_m,  rho_m = e^{-x_m},  x_m = r_m dtt,  dtt = dt lambda^{1/alpha}
//
// The retention rho enters through the decays between tokens, exp(-sum of x over the
// tokens between them).  Differentiating every decay that spans token j by x_j gives
// the telescoped form (derived here; the paper does not state a backward pass):
//
//   d dtt_j = sum_m r_m mu_{j,m} X_m(j) + sum_m r_m rho_{j,m} w_{j,m} dk_{j,m}
//   X_m(j)  = -(sum_{t' = j}^{j2 - 1} g_{t',m}  [+ <dS_final, S_final>_m if j2 = L])
//   g_{t,m} = c_{t,m} dc_{t,m} - kappa_{t,m} dk_{t,m}
//
// where j2 is the first token after j whose exponent x reaches the cut X_cut in mode m
// (L if none) and mu_{j,m} is 1 when x_{j,m} is below it.  Every decay across such a
// token is at most e^{-X_cut}, so what lies beyond it, and the token's own term
// (proportional to that decay), is below the rounding of the path: the sum stops there
// and the term is dropped.  X_cut is 16 for float32 I/O (e^{-16} ~ 1.1e-7) and 8 for
// bfloat16 I/O (e^{-8} ~ 3.4e-4; the matrix-core operands of the state and adjoint
// updates carry 2^-9 relative rounding).  Without the stop, the suffix sum across such
// a token is a difference of terms whose exact value is near zero: each term is
// formed once from the state side (dc) and once from the adjoint side (dk), each
// rounded its own way, and that rounding, multiplied by r_m lambda^{1/alpha} (up to
// 2^100), would swamp ddt.
//
// Then ddt = s d dtt with s = lambda^{1/alpha}, and with ds = ddt dt:
//   dalpha  = -sum_m (dz_c + dz_w)_m ln tau_m - ds ln(lambda) / alpha^2
//   dlambda = ds / (alpha lambda)
//   dz_c = c (dc - sum c dc),  dz_w = w (dw - sum w dw),  dw = beta dk
// (dalpha and dlambda take no step term where the library holds lambda^{1/alpha} at
// 2^100: the held value does not depend on them).
//
// Two kernels, one workgroup of four waves (four heads, lane = token) per 64-token
// tile: the first sums the partials and forms, per mode, the tile's head segment
// (the sum of g from the tile's first token up to its first capped token); the
// second forms the carry from the later tiles' segments, the segmented suffix sums
// inside the tile, and every output.  All sums run in a fixed order.
#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

// Exponent r_m dtt at which a token cuts the per-mode suffix sums (see above).
__device__ __forceinline__ float cut_exponent(const ScanParams& p) { return p.io_bf16 ? 8.0f : 16.0f; }

// The per-token coefficients a lane needs: c, w over all modes, the effective step.
template <int MP>
struct TokenCoef {
  float c[MP], w[MP];
  float dtv, al, lam, s_eff, dtt;
};

// Loads M (<= MP) consecutive floats at p (16-byte aligned when M is a multiple of 4).
template <int MP>
__device__ __forceinline__ void load_modes(const float* p, int M, float* out) {
  if (M == MP && (MP % 4) == 0) {
#pragma unroll
    for (int j = 0; j < MP / 4; ++j) {
      const float4 v = reinterpret_cast<const float4*>(p)[j];
      out[4 * j] = v.x;
      out[4 * j + 1] = v.y;
      out[4 * j + 2] = v.z;
      out[4 * j + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int m = 0; m < MP; ++m) out[m] = (m < M) ? p[m] : 0.0f;
  }
}

template <int MP>
__device__ __forceinline__ void store_modes(float* p, int M, const float* v) {
  if (M == MP && (MP % 4) == 0) {
#pragma unroll
    for (int j = 0; j < MP / 4; ++j)
      reinterpret_cast<float4*>(p)[j] = make_float4(v[4 * j], v[4 * j + 1], v[4 * j + 2], v[4 * j + 3]);
  } else {
#pragma unroll
    for (int m = 0; m < MP; ++m)
      if (m < M) p[m] = v[m];
  }
}

template <int MP>
__device__ __forceinline__ void token_coef(const ScanParams& p, int b, int t, int h, bool valid, const float* s_lnt,
                                           TokenCoef<MP>& k) {
  const int M = p.M;
  const int64_t tok = ((int64_t)b * p.L + t) * p.H + h;
  k.dtv = valid ? p.dt[tok] : 0.0f;
  k.al = valid ? strided3(p.alpha, p.as0, p.as1, p.as2, b, t, h) : 1.0f;
  k.lam = (valid && p.lambda) ? strided3(p.lambda, p.ls0, p.ls1, p.ls2, b, t, h) : 1.0f;
  k.s_eff = p.lambda ? step_factor(k.lam, k.al) : 1.0f;
  k.dtt = k.dtv * k.s_eff;
  float rl[MP], wl[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) rl[m] = wl[m] = 0.0f;
  if (valid && p.read_logit) load_modes<MP>(p.read_logit + tok * M, M, rl);
  if (valid && p.write_logit && p.write_logit != p.read_logit) load_modes<MP>(p.write_logit + tok * M, M, wl);
  const bool same = p.write_logit == p.read_logit;
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    const float prior = -k.al * s_lnt[m];
    k.c[m] = prior + rl[m];
    k.w[m] = prior + (same ? rl[m] : wl[m]);
  }
  softmax_fast<MP>(k.c, M);
  softmax_fast<MP>(k.w, M);
}

// Composition of the maps z -> v_j + a_j z of lanes j .. 63 (a in {0, 1}), as (A, V).
__device__ __forceinline__ void suffix_affine(float& A, float& V) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const float Ad = __shfl_down(A, d, 64), Vd = __shfl_down(V, d, 64);
    if (lane + d < 64) {
      V = V + A * Vd;
      A = A * Ad;
    }
  }
}

// The carry into `tile` from the later tiles of one (batch, head) and mode: the sum
// of their head segments up to the first capped token, the final-state term Fm as
// the segment of a virtual tile after the last.  Wave-uniform.
__device__ __forceinline__ float tile_carry(const float* tileV, const int* tileF, int64_t row, int tile, int ntiles,
                                            int M, int m, float Fm) {
  const int lane = threadIdx.x & 63;
  float sum = 0.0f;
  for (int g0 = tile + 1; g0 <= ntiles; g0 += 64) {
    const int tj = g0 + lane;
    float v = 0.0f;
    int f = 3;  // bit 0: first token below the cap; bit 1: no capped token after it in the tile
    if (tj < ntiles) {
      v = tileV[(row + tj) * M + m];
      f = tileF[(row + tj) * M + m];
    } else if (tj == ntiles) {
      v = Fm;
    }
    // tile j is cut off by its own first token, or by a capped token inside tile j - 1
    const uint64_t self = __ballot(!(f & 1));
    const uint64_t after = __ballot(!(f & 2));
    const uint64_t stop_mask = self | (after << 1);
    const int stop = stop_mask ? __builtin_ctzll(stop_mask) : 64;
    sum += group_allreduce<64>(lane < stop ? v : 0.0f, [](float x, float y) { return x + y; });
    if (stop < 64 || ((after >> 63) & 1)) break;
  }
  return sum;
}

template <int MP>
__global__ void __launch_bounds__(256) frac_grad_tiles_kernel(ScanParams p, GradInputs gi) {
  __shared__ float s_rr[MP], s_lnt[MP];
  if (threadIdx.x < MP) {
    const int m = threadIdx.x;
    const float tau = m < p.M ? p.tau[m] : 1.0f;
    s_rr[m] = m < p.M ? 1.0f / tau : 0.0f;
    s_lnt[m] = m < p.M ? logf(tau) : 0.0f;
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nhq = (p.H + 3) / 4, ntl = (p.L + 63) / 64;
  const int hq = (int)(blockIdx.x % nhq), tile = (int)((blockIdx.x / nhq) % ntl), b = (int)(blockIdx.x / nhq / ntl);
  const int h = hq * 4 + wave;
  if (h >= p.H) return;
  const int L = p.L, M = p.M, ntiles = (L + 63) / 64;
  const int t = tile * 64 + lane;
  const bool valid = t < L;
  TokenCoef<MP> k;
  token_coef<MP>(p, b, valid ? t : L - 1, h, valid, s_lnt, k);
  const int64_t bh = (int64_t)b * p.H + h;
  const int64_t S = (int64_t)p.Bsz * p.H * L * M;
  const int64_t i0 = (bh * L + t) * M;
  float dc[MP], dk[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) dc[m] = dk[m] = 0.0f;
  if (valid) {
    for (int q = 0; q < gi.ndc; ++q) {
      float v[MP];
      load_modes<MP>(gi.dc + q * S + i0, M, v);
#pragma unroll
      for (int m = 0; m < MP; ++m) dc[m] += v[m];
    }
    for (int q = 0; q < gi.ndk; ++q) {
      float v[MP];
      load_modes<MP>(gi.dk + q * S + i0, M, v);
#pragma unroll
      for (int m = 0; m < MP; ++m) dk[m] += v[m];
    }
    store_modes<MP>(gi.dc + i0, M, dc);  // the sums, for the second kernel
    store_modes<MP>(gi.dk + i0, M, dk);
  }
  const int64_t row = bh * ntiles;
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    if (m >= M) continue;  // wave-uniform
    const float x = s_rr[m] * k.dtt;
    const bool capped = valid && !(x < cut_exponent(p));
    const float kap = one_minus_exp_neg(x) * k.w[m];
    const float g = valid ? k.c[m] * dc[m] - kap * dk[m] : 0.0f;
    const uint64_t cb = __ballot(capped);
    const uint64_t after = cb & ~1ull;
    const int fc = after ? __builtin_ctzll(after) : 64;
    const float V = group_allreduce<64>(lane < fc ? g : 0.0f, [](float a, float c) { return a + c; });
    if (lane == 0) {
      gi.tileV[(row + tile) * M + m] = V;
      gi.tileF[(row + tile) * M + m] = (capped ? 0 : 1) | (after ? 0 : 2);
    }
  }
}

template <int MP>
__global__ void __launch_bounds__(256) frac_grad_finish_kernel(ScanParams p, GradInputs gi) {
  __shared__ float s_rr[MP], s_lnt[MP];
  if (threadIdx.x < MP) {
    const int m = threadIdx.x;
    const float tau = m < p.M ? p.tau[m] : 1.0f;
    s_rr[m] = m < p.M ? 1.0f / tau : 0.0f;
    s_lnt[m] = m < p.M ? logf(tau) : 0.0f;
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nhq = (p.H + 3) / 4, ntl = (p.L + 63) / 64;
  const int hq = (int)(blockIdx.x % nhq), tile = (int)((blockIdx.x / nhq) % ntl), b = (int)(blockIdx.x / nhq / ntl);
  const int h = hq * 4 + wave;
  if (h >= p.H) return;
  const int L = p.L, H = p.H, M = p.M, ntiles = (L + 63) / 64;
  const int t = tile * 64 + lane;
  const bool valid = t < L;
  TokenCoef<MP> k;
  token_coef<MP>(p, b, valid ? t : L - 1, h, valid, s_lnt, k);
  const int64_t bh = (int64_t)b * H + h;
  const int64_t i0 = (bh * L + t) * M;
  float dc[MP], dk[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) dc[m] = dk[m] = 0.0f;
  if (valid) {
    load_modes<MP>(gi.dc + i0, M, dc);
    load_modes<MP>(gi.dk + i0, M, dk);
  }
  const int64_t row = bh * ntiles;
  const int64_t SF = (int64_t)p.Bsz * H * M;
  float ddtt = 0.0f, scd = 0.0f, swd = 0.0f;
  float beta[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    beta[m] = 0.0f;
    if (m >= M) continue;  // wave-uniform
    const float r = s_rr[m];
    const float x = r * k.dtt;
    const bool mu = x < cut_exponent(p);
    const float rho = __expf(-x);
    beta[m] = one_minus_exp_neg(x);
    const float kap = beta[m] * k.w[m];
    const float g = valid ? k.c[m] * dc[m] - kap * dk[m] : 0.0f;
    float Fm = 0.0f;
    for (int q = 0; q < gi.nF; ++q) Fm += gi.F[q * SF + bh * M + m];
    const float carry = tile_carry(gi.tileV, gi.tileF, row, tile, ntiles, M, m, Fm);
    // acc_j = g_j + mu_{j+1} acc_{j+1} inside the tile, acc after the last lane = carry
    const float mu_next = __shfl_down(mu ? 1.0f : 0.0f, 1, 64);
    float A = (lane == 63) ? 1.0f : mu_next, V = g;  // tokens past the sequence: mask 1, g 0
    suffix_affine(A, V);
    const float acc = V + A * carry;
    if (valid) {
      ddtt += r * (mu ? -acc : 0.0f) + r * rho * k.w[m] * dk[m];
      scd += k.c[m] * dc[m];
      swd += k.w[m] * (beta[m] * dk[m]);
    }
  }
  const int64_t tok = ((int64_t)b * L + t) * H + h;
  float dap = 0.0f;
  if (valid && (p.dread_logit || p.dwrite_logit || p.dalpha)) {
    float zc[MP], zw[MP];
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      zc[m] = zw[m] = 0.0f;
      if (m >= M) continue;
      zc[m] = k.c[m] * (dc[m] - scd);
      zw[m] = k.w[m] * (beta[m] * dk[m] - swd);
      dap -= (zc[m] + zw[m]) * s_lnt[m];
    }
    if (p.dread_logit) store_modes<MP>(p.dread_logit + tok * M, M, zc);
    if (p.dwrite_logit) store_modes<MP>(p.dwrite_logit + tok * M, M, zw);
  }
  if (valid) {
    const float ddt = ddtt * k.s_eff;
    p.ddt[tok] = ddt;
    // no step term where the factor lambda^{1/alpha} is held at its bound
    const bool held = p.lambda && !(log2f(k.lam) / k.al <= 100.0f);
    const float ds = (p.lambda && !held) ? ddt * k.dtv : 0.0f;
    const float lnl = p.lambda ? logf(k.lam) : 0.0f;
    if (p.dalpha) p.dalpha[tok] = dap + ((ds != 0.0f && lnl != 0.0f) ? -ds * lnl / (k.al * k.al) : 0.0f);
    if (p.dlambda) p.dlambda[tok] = ds != 0.0f ? ds / (k.al * k.lam) : 0.0f;
  }
  if (p.dD && b == 0 && tile == 0 && lane == 0) {
    float acc = 0.0f;
    for (int q = 0; q < gi.nD; ++q)
      for (int bb = 0; bb < p.Bsz; ++bb) acc += gi.dDp[((int64_t)q * p.Bsz + bb) * H + h];
    p.dD[h] = acc;
  }
}

template <int MP>
hipError_t launch_grads_mp(const ScanParams& p, const GradInputs& gi, hipStream_t stream) {
  const int64_t nblk = (int64_t)p.Bsz * ((p.L + 63) / 64) * ((p.H + 3) / 4);
  const dim3 grid((unsigned)nblk);
  hipLaunchKernelGGL((frac_grad_tiles_kernel<MP>), grid, dim3(256), 0, stream, p, gi);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((frac_grad_finish_kernel<MP>), grid, dim3(256), 0, stream, p, gi);
  return hipGetLastError();
}

}  // namespace

size_t grad_tiles_bytes(const ScanParams& p) {
  const size_t n = (size_t)p.Bsz * p.H * ((p.L + 63) / 64) * p.M;
  return n * (sizeof(float) + sizeof(int));
}

hipError_t launch_grad_finish(const ScanParams& p, const GradInputs& gi, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  if (p.M <= 4) return launch_grads_mp<4>(p, gi, stream);
  if (p.M <= 8) return launch_grads_mp<8>(p, gi, stream);
  if (p.M <= 16) return launch_grads_mp<16>(p, gi, stream);
  return launch_grads_mp<32>(p, gi, stream);
}

}  // namespace frac
