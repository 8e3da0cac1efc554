// frac_nfree.hip -- chunked forward scan of the paper's own layer form: no B/C
// projections (B = C = 1), so each head carries an M x d_h state, the recurrence
// of the Appendix-D algorithm (Sec. 3.2, eq. frac-selective-update and
// eq. frac-readout with a scalar write/read), evaluated chunk by chunk as in the
// remark closing Sec. 3.2.  With r_m = 1 / tau_m and A_t the chunk-local inclusive
// sum of the effective steps:
//
//   y_t = sum_m c_{t,m} e^{-r_m A_t} S_m + sum_{k<=t} Gamma_{t,k} x_k + D x_t
//   Gamma_{t,k} = sum_m c_{t,m} kappa_{k,m} e^{-r_m (A_t - A_k)}
//   S_m <- e^{-r_m A_Q} S_m + sum_k kappa_{k,m} e^{-r_m (A_Q - A_k)} x_k
//
// One workgroup of 4 waves per (batch, head, 64 columns of d_h); wave w owns
// columns 16 w .. 16 w + 15 and the state of all modes for them (at most two
// 16x16 float32 accumulator tiles, modes as rows).  Per chunk: x copied into LDS,
// per-(token, mode) weights, Gamma in causal 16x16 tiles (float32 matrix cores,
// modes as K; one exponential per pair for modes whose chunk decay passes the
// factorisation bound), then the readout (weights x state, K = modes), the
// intra-chunk product Gamma x (K = tokens) and the state update (K = tokens) on
// the matrix cores.  The state scale trick of the B/C scan applies unchanged.
#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

__constant__ int kNfTB[10] = {0, 1, 1, 2, 2, 2, 3, 3, 3, 3};
__constant__ int kNfKB[10] = {0, 0, 1, 0, 1, 2, 0, 1, 2, 3};
constexpr float kNfSafe = 55.0f;
constexpr float kNfFloor = 0x1p-60f;


template <typename T, int MP>
__global__ void __launch_bounds__(256) frac_nfree_fwd_kernel(ScanParams p) {
  constexpr bool kBf16 = sizeof(T) == 2;
  constexpr int MB = (MP + 15) / 16;        // 16-row blocks of modes in the state
  constexpr int XS = kBf16 ? 64 + 8 : 64 + 4;  // [t][p] and [t][k] tile strides
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, M = p.M;
  const int nps = (P + 63) / 64;
  const int ps = blockIdx.x % nps, bh = blockIdx.x / nps, b = bh / H, h = bh - b * H;
  const int p0 = ps * 64, pc = p0 + wave * 16 + li;  // this lane's column of d_h
  const bool active = p0 + wave * 16 < P;
  const int nchunks = (L + kQ - 1) / kQ;

  __shared__ __align__(16) T Xs[64 * XS];  // x of the chunk [t][p]
  __shared__ __align__(16) T Gs[64 * XS];  // causal Gamma [t][k]
  __shared__ __align__(16) T Ys[64 * XS];  // output rows [t][p]
  // per-token weight arrays [MP][WQ]: the row stride of 68 floats spreads the
  // stores of one wave (4 tokens x 16 modes, or 8 x 8) over distinct LDS banks
  constexpr int WQ = kQ + 4;
  __shared__ __align__(16) float W[7 * MP * WQ + kQ];
  __shared__ float s_rr[MP], s_lnt[MP], s_E2[2][MP];
  float* P_om = W;                 // [MP][Q] c e^{-rA_t} E_m   (readout)
  float* P_v = W + MP * WQ;        // [MP][Q] kappa e^{-r(A_Q-A_t)} upd (update)
  float* P_O = W + 2 * MP * WQ;    // [MP][Q] c e^{-rA_t}        (Gamma rows)
  float* P_Vt = W + 3 * MP * WQ;   // [MP][Q] kappa e^{rA_t}, safe modes (Gamma columns)
  float* P_c = W + 4 * MP * WQ;    // [MP][Q] c, kappa (modes past the factorisation bound)
  float* P_k = W + 5 * MP * WQ;
  float* P_A = W + 7 * MP * WQ;    // [Q] A_t

  // Gamma tiles above the diagonal that the intra product reads are never written
  for (int i = tid; i < 64 * XS; i += 256) Gs[i] = (T)0.0f;
  if (tid < MP) {
    const float tau = (tid < M) ? p.tau[tid] : 1.0f;
    s_rr[tid] = (tid < M) ? 1.0f / tau : 0.0f;
    s_lnt[tid] = (tid < M) ? logf(tau) : 0.0f;
    s_E2[0][tid] = s_E2[1][tid] = 1.0f;
  }
  // the state: S[mb] holds modes 16 mb + 4 lg + r, column pc
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)M * P;
  floatx4 S[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = mb * 16 + lg * 4 + r;
      S[mb][r] = (p.init_state && active && m < M && pc < P) ? p.init_state[sbase + (int64_t)m * P + pc] : 0.0f;
    }
  const float Dh = p.D ? p.D[h] : 0.0f;

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * P + p0;
  T* yg = reinterpret_cast<T*>(p.y) + (((int64_t)b * L) * H + h) * P + p0;
  const int64_t xstride = (int64_t)H * P;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const int64_t lg_st = (int64_t)H * M;
  constexpr int E16 = 16 / (int)sizeof(T);  // elements per 16-byte vector
  constexpr int CPR = 64 / E16;             // 16-byte vectors per 64-column row
  constexpr int XV = 64 * CPR / 256;        // 16-byte vectors of x per thread and chunk

  // x and the per-token controls of a chunk, loaded one chunk ahead into registers
  int4 xr[XV];
  float dt_n, al_n, lam_n;
  auto prefetch = [&](int c) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
#pragma unroll
    for (int j = 0; j < XV; ++j) {
      const int i = tid + 256 * j, t = i / CPR, col = (i - t * CPR) * E16;
      xr[j] = make_int4(0, 0, 0, 0);
      if (t < nv && p0 + col < P) xr[j] = *reinterpret_cast<const int4*>(xg + (int64_t)(t0 + t) * xstride + col);
    }
    const int tg = t0 + lane;
    const bool tvalid = lane < nv;
    dt_n = tvalid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al_n = tvalid ? al_bh[tg * p.as1] : 1.0f;
    lam_n = (tvalid && lm_bh) ? lm_bh[tg * p.ls1] : 1.0f;
  };
  prefetch(0);

  for (int c = 0; c < nchunks; ++c) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    const float* Ecur = s_E2[c & 1];
    float* Enext = s_E2[(c + 1) & 1];
    __syncthreads();  // the previous chunk is done with every LDS array
    // ---- x of the chunk into LDS (zeros past the sequence and past d_h)
#pragma unroll
    for (int j = 0; j < XV; ++j) {
      const int i = tid + 256 * j, t = i / CPR, col = (i - t * CPR) * E16;
      *reinterpret_cast<int4*>(Xs + t * XS + col) = xr[j];
    }
    const bool tvalid = lane < nv;
    const float dtv = dt_n, al_l = al_n, lam = lam_n;
    if (c + 1 < nchunks) prefetch(c + 1);
    // ---- per-token controls (lane = token, every wave) and their chunk-local sum
    const float s_eff = lm_bh ? exp2f(log2f(lam) / al_l) : 1.0f;
    const float dtt_l = tvalid ? dtv * s_eff : 0.0f;
    const float A_l = wave_inclusive_sum(dtt_l);
    const float Alast = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(A_l), 63));
    if (wave == 0) P_A[lane] = A_l;
    const bool over = lane < MP && lane < M && !(s_rr[lane < MP ? lane : 0] * Alast <= kNfSafe);
    const int unsafe = (int)(__ballot(over) & ((MP >= 32) ? 0xffffffffull : ((1ull << MP) - 1)));
    // ---- per (token, mode) weights: pair = t MP + m
    for (int pr = tid; pr < kQ * MP; pr += 256) {
      const int t = pr / MP, m = pr - t * MP;
      const float A = __shfl(A_l, t, 64), dtt = __shfl(dtt_l, t, 64), al = __shfl(al_l, t, 64);
      const bool valid = t < nv;
      const int64_t ith = (int64_t)(t0 + t) * lg_st + m;
      const float r = s_rr[m], prior = -al * s_lnt[m];
      const float zc = (m < M) ? prior + ((rl_bh && valid) ? rl_bh[ith] : 0.0f) : -INFINITY;
      const float zw = (m < M) ? prior + ((wl_bh && valid) ? wl_bh[ith] : 0.0f) : -INFINITY;
      const float cw = valid ? group_softmax<MP>(zc) : 0.0f;
      const float ww = (rl_bh == wl_bh) ? cw : (valid ? group_softmax<MP>(zw) : 0.0f);
      const float xr = r * Alast;
      const bool safe = xr <= kNfSafe;
      const float Enew = Ecur[m] * fexp(-xr);
      const bool ren = !(Enew >= kNfFloor);
      const float upd = ren ? 1.0f : __frcp_rn(Enew);
      const float kap = one_minus_exp_neg(dtt * r) * ww;
      const float om = cw * fexp(-r * A);
      P_O[m * WQ + t] = om;
      P_om[m * WQ + t] = om * Ecur[m];
      P_v[m * WQ + t] = kap * fexp(-r * (Alast - A)) * upd;
      P_Vt[m * WQ + t] = safe ? kap * fexp(r * A) : 0.0f;
      P_c[m * WQ + t] = cw;
      P_k[m * WQ + t] = kap;
      if (pr < MP) Enext[m] = ren ? 1.0f : Enew;
    }
    float renf[MB * 4];
    bool ren_any = false;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb * 16 + lg * 4 + r;
        const float Enew = (m < MP) ? Ecur[m] * fexp(-s_rr[m] * Alast) : 1.0f;
        renf[mb * 4 + r] = Enew;
        ren_any |= !(Enew >= kNfFloor);
      }
    __syncthreads();  // x and the weights in LDS

    // ---- causal Gamma tiles [t][k] (float32 matrix cores, modes as K)
    for (int tile = wave; tile < 10; tile += 4) {
      const int tb = kNfTB[tile], kb = kNfKB[tile];
      floatx4 Gm = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < (MP + 3) / 4; ++q) {
        const int m = q * 4 + lg;
        const float av = (m < MP) ? P_O[m * WQ + tb * 16 + li] : 0.0f;
        const float bv = (m < MP) ? P_Vt[m * WQ + kb * 16 + li] : 0.0f;
        Gm = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, Gm, 0, 0, 0);
      }
      if (unsafe) {
        for (int m = 0; m < MP; ++m) {
          if (!((unsafe >> m) & 1)) continue;
          const float rm = s_rr[m];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
            if (t >= k) Gm[r] += P_c[m * WQ + t] * P_k[m * WQ + k] * fexp(-rm * (P_A[t] - P_A[k]));
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
        Gs[t * XS + k] = (T)keep_if_ge(Gm[r], t, k);
      }
    }
    __syncthreads();  // Gamma in LDS

    if (active) {
      // ---- readout, intra-chunk product and skip term, 4 row blocks of 16 tokens
      Frag<T> Sf;  // the state as a B operand: slot s < 4 mode 4 lg + s, s >= 4 mode 16 + 4 lg + s - 4
#pragma unroll
      for (int s = 0; s < 4; ++s) frag_set(Sf, s, S[0][s]);
#pragma unroll
      for (int s = 0; s < 4; ++s) frag_set(Sf, 4 + s, MB > 1 ? S[MB - 1][s] : 0.0f);
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        const int t = tb * 16 + li;  // A-operand row
        floatx4 Y = {0.f, 0.f, 0.f, 0.f};
        Frag<T> Of;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const int m0 = lg * 4 + s, m1 = 16 + lg * 4 + s;
          frag_set(Of, s, (m0 < MP) ? P_om[m0 * WQ + t] : 0.0f);
          frag_set(Of, 4 + s, (MB > 1 && m1 < MP) ? P_om[m1 * WQ + t] : 0.0f);
        }
        mma(Y, Of, Sf);
#pragma unroll
        for (int kk = 0; kk <= tb / 2; ++kk) {
          const Frag<T> a = frag_load8(Gs + t * XS + kk * 32 + lg * 8);
          const Frag<T> bx = frag_load_rows(Xs, XS, kk * 32 + lg * 8, wave * 16);
          mma(Y, a, bx);
        }
        float xv[4];
        col4_rows(Xs, XS, tb * 16 + lg * 4, wave * 16, xv);
#pragma unroll
        for (int r = 0; r < 4; ++r) Ys[(tb * 16 + lg * 4 + r) * XS + wave * 16 + li] = (T)(Y[r] + Dh * xv[r]);
      }

      // ---- state update S_m <- (rescale) + V^T x, V = kappa e^{-r(A_Q - A_k)} upd
      if (ren_any) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (!(renf[mb * 4 + r] >= kNfFloor)) S[mb][r] *= renf[mb * 4 + r];
      }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const Frag<T> bx = frag_load_rows(Xs, XS, kt * 32 + lg * 8, wave * 16);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int m = mb * 16 + li;  // A-operand row (mode)
          Frag<T> Vf;
          if (m < MP) {
            const float* pv = P_v + m * WQ + kt * 32 + lg * 8;
            const float4 v0 = *reinterpret_cast<const float4*>(pv);
            const float4 v1 = *reinterpret_cast<const float4*>(pv + 4);
            frag_set(Vf, 0, v0.x);
            frag_set(Vf, 1, v0.y);
            frag_set(Vf, 2, v0.z);
            frag_set(Vf, 3, v0.w);
            frag_set(Vf, 4, v1.x);
            frag_set(Vf, 5, v1.y);
            frag_set(Vf, 6, v1.z);
            frag_set(Vf, 7, v1.w);
          } else {
            Vf = frag_zero<T>();
          }
          mma(S[mb], Vf, bx);
        }
      }
    }
    __syncthreads();  // output rows in LDS
    // ---- output rows -> global, 16 bytes per thread
    for (int i = tid; i < 64 * CPR; i += 256) {
      const int t = i / CPR, ch = i - t * CPR, col = ch * E16;
      if (t < nv && p0 + col < P)
        *reinterpret_cast<int4*>(yg + (int64_t)(t0 + t) * xstride + col) = *reinterpret_cast<const int4*>(Ys + t * XS + col);
    }
  }

  if (p.final_state && active) {
    __syncthreads();
    const float* Ef = s_E2[nchunks & 1];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb * 16 + lg * 4 + r;
        if (m < M && pc < P) p.final_state[sbase + (int64_t)m * P + pc] = S[mb][r] * Ef[m];
      }
  }
}

template <typename T>
hipError_t launch_nfree_t(const ScanParams& p, hipStream_t stream) {
  const unsigned blocks = (unsigned)((int64_t)p.Bsz * p.H * ((p.P + 63) / 64));
  if (p.M <= 4) hipLaunchKernelGGL((frac_nfree_fwd_kernel<T, 4>), dim3(blocks), dim3(256), 0, stream, p);
  else if (p.M <= 8) hipLaunchKernelGGL((frac_nfree_fwd_kernel<T, 8>), dim3(blocks), dim3(256), 0, stream, p);
  else if (p.M <= 16) hipLaunchKernelGGL((frac_nfree_fwd_kernel<T, 16>), dim3(blocks), dim3(256), 0, stream, p);
  else hipLaunchKernelGGL((frac_nfree_fwd_kernel<T, 32>), dim3(blocks), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_nfree_fwd(const ScanParams& p, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  return p.io_bf16 ? launch_nfree_t<bf16>(p, stream) : launch_nfree_t<float>(p, stream);
}

}  // namespace frac
