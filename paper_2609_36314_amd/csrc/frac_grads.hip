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
// (derived here; the paper does not state a backward pass)
//
//   d dtt_j = sum_m r_m mu_{j,m} X_m(j) + sum_m r_m rho_{j,m} w_{j,m} dk_{j,m}
//   X_m(j)  = -R_m(j),   R_m(j) = <rho_{j,m} dS_{j,m}, S_{j-1,m}>
//
// R_m(j) pairs the adjoint carried back across token j with the state carried into
// it.  It is never formed from the states (N x P per token and mode) but from the
// per-(token, mode) partials, in one of three exact forms:
//
//   chunk-local, for j in a chunk C (the 64 tokens of one tile):
//     R_m(j) = e^{-(l_end - l_start)} <G_C, S_C>_m + sum_{k in C, k < j} kappa_k dk^inter_k
//              + sum_{t in C, t >= j} (c_t dc_t - kappa_t dk^intra_t)
//     where dk = dk^inter + dk^intra splits the adjoint at the chunk's end (G_C, carried
//     in from the later chunks) from the chunk's own readouts, S_C is the state before
//     the chunk and l_end - l_start the chunk's total exponent;
//   suffix:  R_m(j) = <dS_final, S_final>_m + sum_{t >= j} g_t
//   prefix:  R_m(j) = <S_init, dS_init>_m - sum_{t < j} g_t,   g_t = c_t dc_t - kappa_t dk_t
//
// Every term of the chunk-local form carries the decay across token j, so the form
// keeps the relative rounding of its terms, but its first term needs the state and
// the adjoint at the chunk boundary together.  Where the chunk's total exponent
// reaches X_cut that term is at most e^{-X_cut} of a pairing and is dropped: such a
// "cut" chunk takes the chunk-local form without it.  The suffix and prefix forms
// telescope: their terms largely cancel (what is written on one side of j and read on
// the same side is not in R), each term is formed once from the state side (dc) and
// once from the adjoint side (dk), each rounded its own way, and r_m lambda^{1/alpha}
// (up to 2^100) multiplies what is left.  They serve the chunks that are not cut, and
// every such sum stops at the nearest cut chunk, whose boundary values the chunk-local
// form gives exactly: sum_{t in C} (c dc - kappa dk^intra) at the first token of a cut
// chunk C, sum_{k in C} kappa dk^inter at the first token after it.  Each token of a
// chunk that is not cut takes the form (suffix or prefix) whose range carries the
// smaller sum of magnitudes |c dc| + |kappa dk|, the rounding of a sum growing with it.
//
// mu_{j,m} is 0 where x_{j,m} itself reaches X_cut: the term is then at most e^{-X_cut}
// of the pairing it scales (and exactly 0 where the exponent is held at its cap).
// X_cut is 16 for float32 I/O (e^{-16} ~ 1.1e-7) and 8 for bfloat16 I/O (e^{-8} ~
// 3.4e-4; the matrix-core operands of the state and adjoint updates carry 2^-9
// relative rounding).  A token at or past the cut lies in a cut chunk.
//
// Then ddt = s d dtt with s = lambda^{1/alpha}, and with ds = ddt dt:
//   dalpha  = -sum_m (dz_c + dz_w)_m ln tau_m - ds ln(lambda) / alpha^2
//   dlambda = ds / (alpha lambda)
//   dz_c = c (dc - sum c dc),  dz_w = w (dw - sum w dw),  dw = beta dk
// (dalpha and dlambda take no step term where the library holds lambda^{1/alpha} at
// 2^100: the held value does not depend on them).
//
// Two kernels, one workgroup of four waves (four heads, lane = token) per 64-token
// tile: the first sums the partials and forms, per mode, whether the tile is cut and
// its two segment values (the sums that the suffix and the prefix forms carry across
// it, with the sums of magnitudes); the second forms the carries from the later and
// the earlier tiles, the sums inside the tile, and every output.  All sums run in a
// fixed order.
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

__device__ __forceinline__ float wave_sum(float v) {
  return group_allreduce<64>(v, [](float x, float y) { return x + y; });
}

template <int CTRL, int ROW_MASK, bool BOUND>
__device__ __forceinline__ float dpp_rows(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xF, BOUND));
}

// Inclusive sum over lanes 0 .. j (row shifts, then the row broadcasts).
__device__ __forceinline__ float wave_prefix_sum(float v) {
  v += dpp_rows<0x111, 0xF, true>(v);   // row_shr:1
  v += dpp_rows<0x112, 0xF, true>(v);   // row_shr:2
  v += dpp_rows<0x114, 0xF, true>(v);   // row_shr:4
  v += dpp_rows<0x118, 0xF, true>(v);   // row_shr:8
  v += dpp_rows<0x142, 0xA, false>(v);  // row_bcast:15
  v += dpp_rows<0x143, 0xC, false>(v);  // row_bcast:31
  return v;
}

// The sums over lanes 0 .. j - 1 (excl) and j .. 63 (suffix) of v.
__device__ __forceinline__ void excl_and_suffix(float v, float& excl, float& suffix) {
  const float inc = wave_prefix_sum(v);
  excl = inc - v;
  suffix = __shfl(inc, 63, 64) - excl;
}

// Composition of the maps z -> v_j + a_j z of lanes j .. 63 (a in {0, 1}), as (A, V, W)
// for two value streams V, W under the same masks.
__device__ __forceinline__ void suffix_affine(float& A, float& V, float& W) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const float Ad = __shfl_down(A, d, 64), Vd = __shfl_down(V, d, 64), Wd = __shfl_down(W, d, 64);
    if (lane + d < 64) {
      V = V + A * Vd;
      W = W + A * Wd;
      A = A * Ad;
    }
  }
}

// Composition of the maps z -> v_j + a_j z of lanes 0 .. j applied in lane order.
__device__ __forceinline__ void prefix_affine(float& A, float& V, float& W) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const float Ad = __shfl_up(A, d, 64), Vd = __shfl_up(V, d, 64), Wd = __shfl_up(W, d, 64);
    if (lane >= d) {
      V = A * Vd + V;
      W = A * Wd + W;
      A = A * Ad;
    }
  }
}

// Per (tile, mode): the value the suffix form carries across the tile (vs) and the
// prefix form (vp), with the sums of magnitudes (ns, np).  A cut tile stops both
// carries and supplies the chunk-local boundary values.
struct TileSeg {
  float vs, ns, vp, np;
};

// The carries into every tile of one (batch, head, mode) row, one wave per row:
//   suffix  C_s(j) = vs_{j+1} + (tile j+1 cut ? 0 : C_s(j+1)),  C_s(last) = <dS_final, S_final>
//   prefix  C_p(j) = vp_{j-1} + (tile j-1 cut ? 0 : C_p(j-1)),  C_p(0) = <S_init, dS_init>
// with the magnitude sums alongside (the anchors count 0), in blocks of 64 tiles.
__global__ void __launch_bounds__(256) frac_grad_carry_kernel(ScanParams p, GradInputs gi) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t rowid = (int64_t)blockIdx.x * 4 + wave;  // (b H + h) M + m
  const int M = p.M, ntiles = (p.L + 63) / 64;
  if (rowid >= (int64_t)p.Bsz * p.H * M) return;
  const int m = (int)(rowid % M);
  const int64_t bh = rowid / M, row = bh * ntiles;
  const int64_t SF = (int64_t)p.Bsz * p.H * M;
  float Fm = 0.0f, Im = 0.0f;
  for (int q = 0; q < gi.nF; ++q) Fm += gi.F[q * SF + rowid];
  for (int q = 0; q < gi.nI; ++q) Im += gi.I[q * SF + rowid];
  const TileSeg* seg = reinterpret_cast<const TileSeg*>(gi.tileV);
  float4* carry = reinterpret_cast<float4*>(gi.carry);
  const int nblk = (ntiles + 63) / 64;
  // suffix, from the last block
  float zv = 0.0f, zn = 0.0f;  // C_s, N_s of the first tile after the block
  for (int kb = nblk - 1; kb >= 0; --kb) {
    const int j = kb * 64 + lane;
    float A = 1.0f, V = 0.0f, W = 0.0f;
    if (j == ntiles - 1) {
      A = 0.0f;
      V = Fm;
    } else if (j < ntiles - 1) {
      const TileSeg sg = seg[(row + j + 1) * M + m];
      A = gi.tileF[(row + j + 1) * M + m] ? 0.0f : 1.0f;
      V = sg.vs;
      W = sg.ns;
    }
    suffix_affine(A, V, W);
    const float cv = V + A * zv, cn = W + A * zn;
    if (j < ntiles) {
      float4& c = carry[(row + j) * M + m];
      c.x = cv;
      c.y = cn;
    }
    zv = __shfl(cv, 0, 64);
    zn = __shfl(cn, 0, 64);
  }
  // prefix, from the first block
  zv = zn = 0.0f;
  for (int kb = 0; kb < nblk; ++kb) {
    const int j = kb * 64 + lane;
    float A = 1.0f, V = 0.0f, W = 0.0f;
    if (j == 0) {
      A = 0.0f;
      V = Im;
    } else if (j < ntiles) {
      const TileSeg sg = seg[(row + j - 1) * M + m];
      A = gi.tileF[(row + j - 1) * M + m] ? 0.0f : 1.0f;
      V = sg.vp;
      W = sg.np;
    }
    prefix_affine(A, V, W);
    const float cv = V + A * zv, cn = W + A * zn;
    if (j < ntiles) {
      float4& c = carry[(row + j) * M + m];
      c.z = cv;
      c.w = cn;
    }
    zv = __shfl(cv, 63, 64);
    zn = __shfl(cn, 63, 64);
  }
}

// Sums the partial slots of one kind for this lane's token into v (zero past the sequence).
template <int MP>
__device__ __forceinline__ void sum_slots(const float* base, int n, int64_t S, int64_t i0, int M, bool valid,
                                          float* v) {
#pragma unroll
  for (int m = 0; m < MP; ++m) v[m] = 0.0f;
  if (!valid) return;
  for (int q = 0; q < n; ++q) {
    float u[MP];
    load_modes<MP>(base + q * S + i0, M, u);
#pragma unroll
    for (int m = 0; m < MP; ++m) v[m] += u[m];
  }
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
  float dc[MP], dkx[MP], dki[MP];
  sum_slots<MP>(gi.dc, gi.ndc, S, i0, M, valid, dc);
  sum_slots<MP>(gi.dk, gi.ndk, S, i0, M, valid, dkx);
  sum_slots<MP>(gi.dki, gi.ndki, S, i0, M, valid, dki);
  if (gi.store_sums && valid) {  // many slots: the sums, for the second kernel
    store_modes<MP>(gi.dc + i0, M, dc);
    store_modes<MP>(gi.dk + i0, M, dkx);
    store_modes<MP>(gi.dki + i0, M, dki);
  }
  const int64_t row = bh * ntiles;
  const float xcut = cut_exponent(p);
  TileSeg* seg = reinterpret_cast<TileSeg*>(gi.tileV);
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    if (m >= M) continue;  // wave-uniform
    const float x = capped_exponent(s_rr[m], k.dtt);
    const bool cut = !(wave_sum(valid ? x : 0.0f) < xcut);
    const float kap = one_minus_exp_neg(x) * k.w[m];
    const float rd = k.c[m] * dc[m], wx = kap * dkx[m], wi = kap * dki[m];
    TileSeg sg;
    if (cut) {
      sg.vs = wave_sum(rd - wi);
      sg.ns = wave_sum(fabsf(rd) + fabsf(wi));
      sg.vp = wave_sum(wx);
      sg.np = wave_sum(fabsf(wx));
    } else {
      const float g = rd - (wx + wi);
      sg.vs = wave_sum(g);
      sg.ns = wave_sum(fabsf(rd) + fabsf(wx + wi));
      sg.vp = -sg.vs;
      sg.np = sg.ns;
    }
    if (lane == 0) {
      seg[(row + tile) * M + m] = sg;
      gi.tileF[(row + tile) * M + m] = cut ? 1 : 0;
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
  const int64_t row = bh * ntiles;
  const float xcut = cut_exponent(p);
  const float4* carry = reinterpret_cast<const float4*>(gi.carry);
  float ddtt = 0.0f, scd = 0.0f, swd = 0.0f;
  float beta[MP];
  {
    // the partial slots summed again in the first kernel's order, or the sums it stored
    const int64_t S = (int64_t)p.Bsz * H * L * M;
    const bool one = gi.store_sums != 0;
    float dkx[MP], dki[MP];
    sum_slots<MP>(gi.dc, one ? 1 : gi.ndc, S, i0, M, valid, dc);
    sum_slots<MP>(gi.dk, one ? 1 : gi.ndk, S, i0, M, valid, dkx);
    sum_slots<MP>(gi.dki, one ? 1 : gi.ndki, S, i0, M, valid, dki);
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      dk[m] = dkx[m] + dki[m];
      beta[m] = 0.0f;
      if (m >= M) continue;  // wave-uniform
      const float r = s_rr[m];
      const float x = capped_exponent(r, k.dtt);
      const bool mu = x < xcut;
      const float rho = __expf(-x);
      beta[m] = one_minus_exp_neg(x);
      const float kap = beta[m] * k.w[m];
      const float rd = k.c[m] * dc[m], wx = kap * dkx[m], wi = kap * dki[m];
      float R, e0, s0;
      if (gi.tileF[(row + tile) * M + m]) {  // cut tile: the chunk-local form
        float e1, s1;
        excl_and_suffix(wx, e0, s0);
        excl_and_suffix(rd - wi, e1, s1);
        R = e0 + s1;
      } else {  // the suffix or the prefix form, whichever range carries less magnitude
        const float4 cr = carry[(row + tile) * M + m];
        const float g = rd - (wx + wi), a = fabsf(rd) + fabsf(wx + wi);
        float e1, s1;
        excl_and_suffix(g, e0, s0);
        excl_and_suffix(a, e1, s1);
        const float rs = cr.x + s0, ns = cr.y + s1;
        const float rp = cr.z - e0, np = cr.w + e1;
        R = (np < ns) ? rp : rs;
      }
      if (valid) {
        ddtt += r * (mu ? -R : 0.0f) + r * rho * k.w[m] * dk[m];
        scd += k.c[m] * dc[m];
        swd += k.w[m] * (beta[m] * dk[m]);
      }
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
hipError_t launch_grads_mp(const ScanParams& p, const GradInputs& gi0, hipStream_t stream) {
  GradInputs gi = gi0;
  // with many partial slots, writing their sums once costs less than reading them twice
  gi.store_sums = gi.ndc + gi.ndk + gi.ndki > 6;
  const int64_t nblk = (int64_t)p.Bsz * ((p.L + 63) / 64) * ((p.H + 3) / 4);
  const dim3 grid((unsigned)nblk);
  hipLaunchKernelGGL((frac_grad_tiles_kernel<MP>), grid, dim3(256), 0, stream, p, gi);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t rows = (int64_t)p.Bsz * p.H * p.M;
  hipLaunchKernelGGL(frac_grad_carry_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, p, gi);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((frac_grad_finish_kernel<MP>), grid, dim3(256), 0, stream, p, gi);
  return hipGetLastError();
}

}  // namespace

size_t grad_tiles_bytes(const ScanParams& p) {
  const size_t n = (size_t)p.Bsz * p.H * ((p.L + 63) / 64) * p.M;
  return n * (sizeof(TileSeg) + sizeof(float4) + sizeof(int));
}

void grad_tiles_at(const ScanParams& p, void* base, GradInputs& gi) {
  const size_t n = (size_t)p.Bsz * p.H * ((p.L + 63) / 64) * p.M;
  unsigned char* at = reinterpret_cast<unsigned char*>(base);
  gi.tileV = reinterpret_cast<float*>(at);
  gi.carry = reinterpret_cast<float*>(at + n * sizeof(TileSeg));
  gi.tileF = reinterpret_cast<int*>(at + n * (sizeof(TileSeg) + sizeof(float4)));
}

hipError_t launch_grad_finish(const ScanParams& p, const GradInputs& gi, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  if (p.M <= 4) return launch_grads_mp<4>(p, gi, stream);
  if (p.M <= 8) return launch_grads_mp<8>(p, gi, stream);
  if (p.M <= 16) return launch_grads_mp<16>(p, gi, stream);
  return launch_grads_mp<32>(p, gi, stream);
}

}  // namespace frac
