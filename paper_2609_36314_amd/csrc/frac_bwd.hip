// frac_bwd.hip -- chunked parallel scan, backward (training).
//
// Reverse-mode derivative of the selective mode-bank recurrence of Sec. 3.2
// (eq. frac-selective-update, eq. frac-readout, the Appendix-D algorithm), with
// the B/C-widened state, evaluated chunk by chunk like the forward.  Per mode
// (r = 1/tau_m), chunk-local inclusive cumulative step A_t, chunk total A_Q,
// state entering the chunk S0 and adjoint of the chunk's last state G_out:
//
//   dC_t  = sum_m c e^{-rA_t} S0^T-contraction: sum_m c_{t,m} e^{-r A_t} S0_m dy_t
//           + sum_{k<=t} Gamma_{t,k} (dy_t . x_k) B_k
//   dx_t  = sum_m kappa_{t,m} e^{-r(A_Q - A_t)} G_out,m^T B_t
//           + sum_{t'>=t} Gamma_{t',t} (C_t' . B_t) dy_t' + D dy_t
//   dB_t  = sum_m kappa_{t,m} e^{-r(A_Q - A_t)} G_out,m x_t
//           + sum_{t'>=t} Gamma_{t',t} (dy_t' . x_t) C_t'
//   G_out(previous chunk) = e^{-r A_Q} G_out + sum_t c_{t,m} e^{-r A_t} C_t dy_t^T
//
// and for the step sizes (with dc = C^T S dy, dkappa = B^T G x per token and mode):
//   ddtt_t = -sum_m r_m <dS_final, S_final>_m - sum_{t'>=t} e_t' + f_t
//   e_t = sum_m r_m (c dc - kappa dkappa)_{t,m},  f_t = sum_m r_m w rho dkappa_{t,m}
//   ddt_t = ddtt_t * lambda_t^(1/alpha_t)
// (the gradient of the cumulative log-retention telescopes into the suffix sum of
// e; derived from the recurrence, checked against the float64 oracle).  Inside a
// chunk the e/f terms reduce to row and column sums of
//   H o Phi and H o Psi,  H = (C B^T) o (dY X^T),
//   Phi_{t,k} = sum_m r_m c_{t,m} kappa_{k,m} e^{-r(A_t - A_k)},
//   Psi_{t,k} = sum_m r_m c_{t,m} w_{k,m} rho_{k,m} e^{-r(A_t - A_k)},
// rank-M products like Gamma.
//
// Three independent sweeps run in one launch (blockIdx.y), one workgroup per
// (batch, head) each; a state or adjoint share lives in matrix-core accumulators:
//   0  forward sweep, state held transposed (wave = 16 columns of N, all of P):
//      recomputes S, gives dC (per head), the readout and intra-chunk parts of
//      e, f, the final-state term and sum(dy . x) for dD;
//   1  reverse sweep, adjoint in row layout (waves = P blocks x N halves): dx and
//      the state-adjoint parts of e and f;
//   2  reverse sweep, adjoint transposed (wave = 16 columns of N): dB (per head).
// A finishing kernel forms ddt from the suffix sums, and a reduction kernel sums
// dB and dC over the heads of each group in a fixed order.
#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

__constant__ int kTB[10] = {0, 1, 1, 2, 2, 2, 3, 3, 3, 3};
__constant__ int kKB[10] = {0, 0, 1, 0, 1, 2, 0, 1, 2, 3};
constexpr int kTiles = 10;
constexpr int kTileElems = 256;
// row block of lower-triangular tile `tile` (0..9, row-major over tb >= kb)
__host__ __device__ constexpr int tile_tb(int tile) { return tile < 1 ? 0 : tile < 3 ? 1 : tile < 6 ? 2 : 3; }
constexpr float kSafeExponent = 55.0f;
constexpr float kRescaleFloor = 0x1p-60f;
constexpr int kPBM = 4;  // p-blocks of 16 held per wave in the transposed layouts (P <= 64)
constexpr int LDQ = kQ + 8;
constexpr int LDP = 64 + 8;

__device__ __forceinline__ float uniform(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

// Sum over the 16 lanes of a lane group of v[j], returned in the lane whose
// index within the group is j (8 + 4 + 2 + 1 exchanges).
__device__ __forceinline__ float transpose_reduce16(float v[16], int li) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const bool hi = li & 8;
    const float send = hi ? v[j] : v[j + 8];
    const float keep = hi ? v[j + 8] : v[j];
    v[j] = keep + __shfl_xor(send, 8, 64);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bool hi = li & 4;
    const float send = hi ? v[j] : v[j + 4];
    const float keep = hi ? v[j + 4] : v[j];
    v[j] = keep + __shfl_xor(send, 4, 64);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const bool hi = li & 2;
    const float send = hi ? v[j] : v[j + 2];
    const float keep = hi ? v[j + 2] : v[j];
    v[j] = keep + __shfl_xor(send, 2, 64);
  }
  {
    const bool hi = li & 1;
    const float send = hi ? v[0] : v[1];
    const float keep = hi ? v[1] : v[0];
    v[0] = keep + __shfl_xor(send, 1, 64);
  }
  return v[0];
}

// Sum over the 16 lanes of a lane group of v[r] (r = 0..3); returned in every
// lane whose index within the group has ((li >> 2) & 3) == r.
__device__ __forceinline__ float reduce16_4(float v[4], int li) {
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const bool hi = li & 8;
    const float send = hi ? v[j] : v[j + 2];
    const float keep = hi ? v[j + 2] : v[j];
    v[j] = keep + __shfl_xor(send, 8, 64);
  }
  {
    const bool hi = li & 4;
    const float send = hi ? v[0] : v[1];
    const float keep = hi ? v[1] : v[0];
    v[0] = keep + __shfl_xor(send, 4, 64);
  }
  v[0] += __shfl_xor(v[0], 2, 64);
  v[0] += __shfl_xor(v[0], 1, 64);
  return v[0];
}

// token of value index j = 4 tb + r held by lane group lg
__device__ __forceinline__ int tok_of(int j, int lg) { return (j >> 2) * 16 + lg * 4 + (j & 3); }

// Stage 64 rows (tokens) of `ncols` io elements, row t at g + t * stride, into
// LDS: natural [t][ldn] and/or transposed [col][LDQ]; rows >= nv and columns
// >= ncols (up to ncols_pad) are zero.
template <typename T>
__device__ __forceinline__ void stage(const T* g, int64_t stride, int ncols, int ncols_pad, int nv, T* nat, int ldn, T* tr) {
  const int groups = ncols_pad >> 3;
  for (int idx = threadIdx.x; idx < kQ * groups; idx += blockDim.x) {
    const int t = idx / groups, c0 = (idx - t * groups) * 8;
    float v[8];
    if (t < nv && c0 < ncols) load8(g + t * stride + c0, v);
    else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = 0.0f;
    }
    if (nat) {
#pragma unroll
      for (int j = 0; j < 8; ++j) nat[t * ldn + c0 + j] = (T)v[j];
    }
    if (tr) {
#pragma unroll
      for (int j = 0; j < 8; ++j) tr[(c0 + j) * LDQ + t] = (T)v[j];
    }
  }
}

// Controls of the lane's token: effective step and the read / write weights.
template <int MP>
__device__ __forceinline__ void token_controls(const ScanParams& p, int b, int h, int64_t tg, bool valid,
                                               const float* lnt, float& dtt, float& s_eff, float* c, float* w) {
  const int64_t ith = ((int64_t)b * p.L + tg) * p.H + h;
  const float dtv = valid ? p.dt[ith] : 0.0f;
  const float al = valid ? strided3(p.alpha, p.as0, p.as1, p.as2, b, tg, h) : 1.0f;
  const float lam = (valid && p.lambda) ? strided3(p.lambda, p.ls0, p.ls1, p.ls2, b, tg, h) : 1.0f;
  s_eff = p.lambda ? exp2f(log2f(lam) / al) : 1.0f;
  dtt = valid ? dtv * s_eff : 0.0f;
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    const float prior = -al * lnt[m];
    c[m] = prior + ((p.read_logit && valid && m < p.M) ? p.read_logit[ith * p.M + m] : 0.0f);
    w[m] = prior + ((p.write_logit && valid && m < p.M) ? p.write_logit[ith * p.M + m] : 0.0f);
  }
  softmax_modes<MP>(c, p.M);
  softmax_modes<MP>(w, p.M);
}

// Per-mode chunk scalars of the lazily rescaled state / adjoint S = E S^:
// this chunk's decay folds into E unless E would drop below the floor, in which
// case the accumulators are rescaled (ren) and E restarts at 1.
struct ModeScale {
  float E;       // scale of the state entering the chunk
  float Enew;    // E * e^{-r A_Q}
  bool ren;      // rescale the accumulators by Enew before adding this chunk
  float upd;     // factor on this chunk's additions (1/Enew or 1)
  bool safe;     // r A_Q small enough for the factorised decay
};

__device__ __forceinline__ void mode_scale(ModeScale& s, float r, float Alast) {
  const float xr = r * Alast;
  s.safe = xr <= kSafeExponent;
  s.Enew = uniform(s.E * expf(-xr));
  s.ren = !(s.Enew >= kRescaleFloor);
  s.upd = s.ren ? 1.0f : 1.0f / s.Enew;
}

__device__ __forceinline__ void mode_scale_advance(ModeScale& s) { s.E = s.ren ? 1.0f : s.Enew; }

// Rank-M product sum_m a[m][row] b[m][col] over a 16x16 tile (float32 matrix cores).
template <int MP>
__device__ __forceinline__ floatx4 rank_m_tile(const float* a, const float* bm, int row0, int col0, int li, int lg) {
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < (MP + 3) / 4; ++q) {
    const int m = q * 4 + lg;
    const float av = (m < MP) ? a[m * kQ + row0 + li] : 0.0f;
    const float bv = (m < MP) ? bm[m * kQ + col0 + li] : 0.0f;
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
  }
  return acc;
}

// dY X^T tile (rows tb, cols kb), K over P (<= 64) from natural-layout LDS.
template <typename T>
__device__ __forceinline__ floatx4 dyx_tile(const T* dYs, const T* Xs, int tb, int kb, int PP, int li, int lg) {
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int p0 = kk * 32 + lg * 8;
    Frag<T> a = frag_zero<T>(), bb = frag_zero<T>();
    if (p0 < PP) {
      a = frag_load8(dYs + (tb * 16 + li) * LDP + p0);
      bb = frag_load8(Xs + (kb * 16 + li) * LDP + p0);
    }
    mma(acc, a, bb);
  }
  return acc;
}

template <typename T>
__device__ __forceinline__ void load_gtile(const T* gt, int tile, int lane, float* Gt) {
#pragma unroll
  for (int r = 0; r < 4; ++r) Gt[r] = to_f32(gt[tile * kTileElems + lane * 4 + r]);
}

// --------------------------------------------------------------------------
// sweep 0: forward direction, state transposed (rows p, columns n)

template <typename T, int MP, int NB>
__device__ __forceinline__ void sweep_state(const ScanParams& p, int b, int h, int g, const T* __restrict__ gtiles,
                            T* __restrict__ dCp, float* __restrict__ eA, float* __restrict__ fA,
                            float* __restrict__ Fw, float* __restrict__ dDp, unsigned char* smem) {
  constexpr int NP = NB * 16;
  const int PP = p.PP, PB = PP / 16, KP = (PB + 1) / 2;
  const int NWT = blockDim.x >> 6;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const bool active = wave < NB;
  const int ncol = wave * 16 + li;  // state column n of this lane
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M;
  const int nchunks = (L + kQ - 1) / kQ;

  T* Xs = reinterpret_cast<T*>(smem);  // [Q][LDP]
  T* XT = Xs + kQ * LDP;               // [64][LDQ]
  T* dYs = XT + 64 * LDQ;              // [Q][LDP]
  T* BT = dYs + kQ * LDP;              // [NP][LDQ]
  T* CT = BT + NP * LDQ;               // [NP][LDQ]
  T* HG = CT + NP * LDQ;               // [Q][LDQ]  Gamma o dY X^T (natural)
  float* P_O = reinterpret_cast<float*>(HG + kQ * LDQ);  // [MP][Q] c e^{-rA}
  float* P_Vt = P_O + MP * kQ;    // kappa e^{rA} (safe)
  float* P_rO = P_Vt + MP * kQ;   // r c e^{-rA}
  float* P_Y = P_rO + MP * kQ;    // r w rho e^{rA} (safe)
  float* P_wdc = P_Y + MP * kQ;   // c e^{-rA} E
  float* P_wec = P_wdc + MP * kQ; // r c e^{-rA} E
  float* P_v = P_wec + MP * kQ;   // kappa e^{-r(A_Q - A)} * upd
  float* P_c = P_v + MP * kQ;     // c
  float* P_k = P_c + MP * kQ;     // kappa
  float* P_wr = P_k + MP * kQ;    // r w rho
  float* P_A = P_wr + MP * kQ;    // [Q]
  float* redR = P_A + kQ;         // [8][Q]  per-wave readout-side partials (also the final reduce)
  float* redC = redR + 8 * kQ;    // [8][Q]  final reduce
  float* slotR = redC + 8 * kQ;   // [10 tiles][16] row sums of H o Phi
  float* slotC = slotR + kTiles * 16;  // column sums of H o Phi
  float* slotF = slotC + kTiles * 16;  // column sums of H o Psi

  float rr[MP], lnt[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    const float tau = (m < M) ? p.tau[m] : 1.0f;
    rr[m] = (m < M) ? 1.0f / tau : 0.0f;
    lnt[m] = (m < M) ? logf(tau) : 0.0f;
  }
  for (int i = tid; i < kQ * LDQ; i += blockDim.x) HG[i] = (T)0.0f;

  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)M * N * P;
  floatx4 S[MP][kPBM];
  ModeScale ms[MP];
  {
    int lo = (lg * 4) * 1 + ncol * P;  // element (n = ncol, p = 16 pb + 4 lg + r) at sbase + m N P + lo + 16 pb + r
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      ms[m].E = 1.0f;
#pragma unroll
      for (int pb = 0; pb < kPBM; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pr = pb * 16 + lg * 4 + r;
          float v = 0.0f;
          if (p.init_state && active && m < M && ncol < N && pr < P)
            v = p.init_state[sbase + (int64_t)m * N * P + lo + pb * 16 + r];
          S[m][pb][r] = v;
        }
    }
  }
  float dd_acc = 0.0f;

  for (int c = 0; c < nchunks; ++c) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    __syncthreads();
    const int64_t xrow0 = (((int64_t)b * L + t0) * H + h) * P;
    const int64_t brow0 = (((int64_t)b * L + t0) * p.G + g) * N;
    stage<T>(reinterpret_cast<const T*>(p.x) + xrow0, (int64_t)H * P, P, PP, nv, Xs, LDP, XT);
    stage<T>(reinterpret_cast<const T*>(p.dy) + xrow0, (int64_t)H * P, P, PP, nv, dYs, LDP, nullptr);
    stage<T>(reinterpret_cast<const T*>(p.Bm) + brow0, (int64_t)p.G * N, N, NP, nv, nullptr, 0, BT);
    stage<T>(reinterpret_cast<const T*>(p.Cm) + brow0, (int64_t)p.G * N, N, NP, nv, nullptr, 0, CT);
    {
      const int t = lane;
      const bool valid = t < nv;
      float dtt, s_eff, cw[MP], ww[MP];
      token_controls<MP>(p, b, h, t0 + t, valid, lnt, dtt, s_eff, cw, ww);
      const float A = wave_inclusive_sum(dtt);
      const float Alast = uniform(__shfl(A, 63, 64));
      if (wave == 0) P_A[t] = A;
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        mode_scale(ms[m], rr[m], Alast);
        if ((m % NWT) != wave) continue;
        const float rho = expf(-dtt * rr[m]);
        const float kap = -expm1f(-dtt * rr[m]) * ww[m];
        const float ea = expf(-rr[m] * A);
        const float ep = ms[m].safe ? expf(rr[m] * A) : 0.0f;
        P_O[m * kQ + t] = cw[m] * ea;
        P_Vt[m * kQ + t] = kap * ep;
        P_rO[m * kQ + t] = rr[m] * cw[m] * ea;
        P_Y[m * kQ + t] = rr[m] * ww[m] * rho * ep;
        P_wdc[m * kQ + t] = cw[m] * ea * ms[m].E;
        P_wec[m * kQ + t] = rr[m] * cw[m] * ea * ms[m].E;
        P_v[m * kQ + t] = kap * expf(-rr[m] * (Alast - A)) * ms[m].upd;
        P_c[m * kQ + t] = cw[m];
        P_k[m * kQ + t] = kap;
        P_wr[m * kQ + t] = rr[m] * ww[m] * rho;
      }
    }
    __syncthreads();

    // sum(dy . x) of the chunk for dD (fixed element assignment per thread)
    for (int i = tid; i < kQ * PP; i += blockDim.x) {
      const int t = i / PP, pc = i - t * PP;
      dd_acc += to_f32(Xs[t * LDP + pc]) * to_f32(dYs[t * LDP + pc]);
    }

    float rowacc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) rowacc[j] = 0.0f;
    // ---- readout-side terms from the state entering the chunk: dC (inter) and e (inter)
    floatx4 dCacc[4];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) dCacc[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (active) {
      Frag<T> Af[4][2];
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int kp = 0; kp < 2; ++kp) {
          Af[tb][kp] = frag_zero<T>();
          if (kp < KP) {
            const T* row = dYs + (tb * 16 + li) * LDP + kp * 32 + lg * 4;
            Af[tb][kp] = frag_load4x2(row, (2 * kp + 1 < PB) ? row + 16 : nullptr);
          }
        }
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (m >= M) continue;
        Frag<T> Sf[2];
#pragma unroll
        for (int kp = 0; kp < 2; ++kp) {
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Sf[kp], s, S[m][2 * kp][s]);
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Sf[kp], 4 + s, S[m][2 * kp + 1][s]);
        }
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
          floatx4 U = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kp = 0; kp < 2; ++kp)
            if (kp < KP) mma(U, Af[tb][kp], Sf[kp]);
          const float4 wd = *reinterpret_cast<const float4*>(P_wdc + m * kQ + tb * 16 + lg * 4);
          const float4 we = *reinterpret_cast<const float4*>(P_wec + m * kQ + tb * 16 + lg * 4);
          dCacc[tb][0] += wd.x * U[0];
          dCacc[tb][1] += wd.y * U[1];
          dCacc[tb][2] += wd.z * U[2];
          dCacc[tb][3] += wd.w * U[3];
          const T* cr = CT + ncol * LDQ + tb * 16 + lg * 4;
          rowacc[tb * 4 + 0] += we.x * U[0] * to_f32(cr[0]);
          rowacc[tb * 4 + 1] += we.y * U[1] * to_f32(cr[1]);
          rowacc[tb * 4 + 2] += we.z * U[2] * to_f32(cr[2]);
          rowacc[tb * 4 + 3] += we.w * U[3] * to_f32(cr[3]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // ---- intra-chunk tiles: HG = Gamma o D (LDS), H o Phi row / column sums, H o Psi column sums
    {
      const T* gt = gtiles + (((int64_t)b * nchunks + c) * p.G + g) * (kTiles * kTileElems);
      for (int tile = wave; tile < kTiles; tile += NWT) {
        const int tb = kTB[tile], kb = kKB[tile];
        float Gt[4];
        load_gtile(gt, tile, lane, Gt);
        const floatx4 D = dyx_tile<T>(dYs, Xs, tb, kb, PP, li, lg);
        floatx4 Gm = rank_m_tile<MP>(P_O, P_Vt, tb * 16, kb * 16, li, lg);
        floatx4 Ph = rank_m_tile<MP>(P_rO, P_Vt, tb * 16, kb * 16, li, lg);
        floatx4 Ps = rank_m_tile<MP>(P_O, P_Y, tb * 16, kb * 16, li, lg);
#pragma unroll
        for (int m = 0; m < MP; ++m) {
          if (ms[m].safe || m >= M) continue;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
            if (t >= k) {
              const float d = P_c[m * kQ + t] * expf(-rr[m] * (P_A[t] - P_A[k]));
              Gm[r] += d * P_k[m * kQ + k];
              Ph[r] += rr[m] * d * P_k[m * kQ + k];
              Ps[r] += d * P_wr[m * kQ + k];
            }
          }
        }
        float rv[4], ce = 0.f, cf = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
          const bool ok = t >= k;
          const float hm = ok ? Gt[r] * D[r] : 0.0f;
          HG[t * LDQ + k] = (T)(ok ? Gm[r] * D[r] : 0.0f);
          rv[r] = hm * Ph[r];
          ce += hm * Ph[r];
          cf += hm * Ps[r];
        }
        const float rs = reduce16_4(rv, li);
        if ((li & 3) == 0) slotR[tile * 16 + lg * 4 + ((li >> 2) & 3)] = rs;
        ce += __shfl_xor(ce, 16, 64);
        ce += __shfl_xor(ce, 32, 64);
        cf += __shfl_xor(cf, 16, 64);
        cf += __shfl_xor(cf, 32, 64);
        if (lg == 0) {
          slotC[tile * 16 + li] = ce;
          slotF[tile * 16 + li] = cf;
        }
      }
    }

    // per-token partials of this wave (readout side) -> LDS
    redR[wave * kQ + tok_of(li, lg)] = transpose_reduce16(rowacc, li);
    __syncthreads();  // HG and the per-wave partials are complete

    if (wave == 0) {
      // token t: readout side (all waves) + row sums of its row-block tiles - column
      // sums of its column-block tiles, in a fixed order
      const int t = lane, tbt = t >> 4, tr = t & 15;
      float er = 0.f, ec = 0.f, ef = 0.f;
      for (int w2 = 0; w2 < NWT; ++w2) er += redR[w2 * kQ + t];
      for (int kb2 = 0; kb2 <= tbt; ++kb2) er += slotR[(tbt * (tbt + 1) / 2 + kb2) * 16 + tr];
      for (int tb2 = tbt; tb2 < 4; ++tb2) {
        ec += slotC[(tb2 * (tb2 + 1) / 2 + tbt) * 16 + tr];
        ef += slotF[(tb2 * (tb2 + 1) / 2 + tbt) * 16 + tr];
      }
      if (t < nv) {
        const int64_t ith = ((int64_t)b * L + t0 + t) * H + h;
        eA[ith] = er - ec;
        fA[ith] = ef;
      }
    }

    if (active) {
      // ---- dC intra: (Gamma o dY X^T) B, causal
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int kk = 0; kk <= tb / 2; ++kk) {
          const Frag<T> a = frag_load8(HG + (tb * 16 + li) * LDQ + kk * 32 + lg * 8);
          const Frag<T> bb = frag_load8(BT + ncol * LDQ + kk * 32 + lg * 8);
          mma(dCacc[tb], a, bb);
        }
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r;
          if (t < nv && ncol < N) dCp[(((int64_t)b * L + t0 + t) * H + h) * N + ncol] = (T)dCacc[tb][r];
        }

      // ---- state update S^T += X^T (v o B), rows p, columns n
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (!ms[m].ren) continue;
#pragma unroll
        for (int pb = 0; pb < kPBM; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) S[m][pb][r] *= ms[m].Enew;
      }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        float br8[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) br8[s] = to_f32(BT[ncol * LDQ + kt * 32 + lg * 8 + s]);
        Frag<T> Bf[MP];
#pragma unroll
        for (int m = 0; m < MP; ++m) {
          const float4 v0 = *reinterpret_cast<const float4*>(P_v + m * kQ + kt * 32 + lg * 8);
          const float4 v1 = *reinterpret_cast<const float4*>(P_v + m * kQ + kt * 32 + lg * 8 + 4);
          frag_set(Bf[m], 0, br8[0] * v0.x);
          frag_set(Bf[m], 1, br8[1] * v0.y);
          frag_set(Bf[m], 2, br8[2] * v0.z);
          frag_set(Bf[m], 3, br8[3] * v0.w);
          frag_set(Bf[m], 4, br8[4] * v1.x);
          frag_set(Bf[m], 5, br8[5] * v1.y);
          frag_set(Bf[m], 6, br8[6] * v1.z);
          frag_set(Bf[m], 7, br8[7] * v1.w);
        }
#pragma unroll
        for (int pb = 0; pb < kPBM; ++pb) {
          if (pb >= PB) continue;
          const Frag<T> a = frag_load8(XT + (pb * 16 + li) * LDQ + kt * 32 + lg * 8);
#pragma unroll
          for (int m = 0; m < MP; ++m)
            if (m < M) mma(S[m][pb], a, Bf[m]);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < MP; ++m) mode_scale_advance(ms[m]);
  }

  // ---- final-state term sum_m r_m <dS_final_m, S_final_m> and sum(dy . x)
  float fpart = 0.0f;
  if (p.d_final_state && active) {
    int lo = ncol * P + lg * 4;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MP; ++m)
#pragma unroll
      for (int pb = 0; pb < kPBM; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pr = pb * 16 + lg * 4 + r;
          if (m < M && ncol < N && pr < P)
            fpart += rr[m] * ms[m].E * S[m][pb][r] *
                     p.d_final_state[sbase + (int64_t)m * N * P + lo + pb * 16 + r];
        }
  }
  __syncthreads();
  redR[tid] = fpart;
  redC[tid] = dd_acc;
  __syncthreads();
  if (tid == 0) {
    float fs = 0.f, ds = 0.f;
    for (int i = 0; i < (int)blockDim.x; ++i) {
      fs += redR[i];
      ds += redC[i];
    }
    Fw[(int64_t)b * H + h] = fs;
    dDp[(int64_t)b * H + h] = ds;
  }
}

// --------------------------------------------------------------------------
// sweep 1: reverse direction, adjoint in row layout (rows n, columns p): dx, e/f adjoint parts

template <typename T, int MP, int NB>
__device__ __forceinline__ void sweep_adj_rows(const ScanParams& p, int b, int h, int g, const T* __restrict__ gtiles,
                               float* __restrict__ eB, float* __restrict__ fB, unsigned char* smem) {
  constexpr int NP = NB * 16;
  constexpr int NH = NB >= 2 ? 2 : 1;
  constexpr int NBW = NB / NH;
  constexpr int KBW = (NBW + 1) / 2;
  constexpr int LDN = NP + 8;
  const int PP = p.PP, NW = PP / 16;
  const int NWT = blockDim.x >> 6;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const bool active = wave < NW * NH;
  const int pb = wave % NW, nh = active ? wave / NW : 0;
  const int pc = pb * 16 + li;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M;
  const int nchunks = (L + kQ - 1) / kQ;

  T* Bs = reinterpret_cast<T*>(smem);  // [Q][LDN]
  T* CT = Bs + kQ * LDN;               // [NP][LDQ]
  T* dYT = CT + NP * LDQ;              // [64][LDQ]
  T* XT = dYT + 64 * LDQ;              // [64][LDQ]
  T* GGT = XT + 64 * LDQ;              // [Q][LDQ]  ((C B^T) o Gamma)^T
  float* P_O = reinterpret_cast<float*>(GGT + kQ * LDQ);
  float* P_Vt = P_O + MP * kQ;
  float* P_c = P_Vt + MP * kQ;
  float* P_k = P_c + MP * kQ;
  float* P_wdx = P_k + MP * kQ;   // kappa e^{-r(A_Q - A)} E
  float* P_wek = P_wdx + MP * kQ; // r kappa e^{-r(A_Q - A)} E
  float* P_wfk = P_wek + MP * kQ; // r w rho e^{-r(A_Q - A)} E
  float* P_om = P_wfk + MP * kQ;  // c e^{-rA} * upd
  float* P_A = P_om + MP * kQ;
  float* YX = P_A + kQ;           // [4 p-blocks][2][2][4][64]
  float* redE = YX + 4 * 1024;    // [NWT][Q]
  float* redF = redE + 8 * kQ;    // [NWT][Q]

  float rr[MP], lnt[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    const float tau = (m < M) ? p.tau[m] : 1.0f;
    rr[m] = (m < M) ? 1.0f / tau : 0.0f;
    lnt[m] = (m < M) ? logf(tau) : 0.0f;
  }
  for (int i = tid; i < kQ * LDQ; i += blockDim.x) GGT[i] = (T)0.0f;

  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)M * N * P;
  floatx4 Gs[MP][NBW];
  ModeScale ms[MP];
  {
    int lo = (nh * NBW * 16 + lg * 4) * P + pc;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      ms[m].E = 1.0f;
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = (nh * NBW + jb) * 16 + lg * 4 + r;
          float v = 0.0f;
          if (p.d_final_state && active && m < M && n < N && pc < P)
            v = p.d_final_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * P];
          Gs[m][jb][r] = v;
        }
    }
  }
  const float Dh = p.D ? p.D[h] : 0.0f;

  for (int c = nchunks - 1; c >= 0; --c) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    __syncthreads();
    const int64_t xrow0 = (((int64_t)b * L + t0) * H + h) * P;
    const int64_t brow0 = (((int64_t)b * L + t0) * p.G + g) * N;
    stage<T>(reinterpret_cast<const T*>(p.Bm) + brow0, (int64_t)p.G * N, N, NP, nv, Bs, LDN, nullptr);
    stage<T>(reinterpret_cast<const T*>(p.Cm) + brow0, (int64_t)p.G * N, N, NP, nv, nullptr, 0, CT);
    stage<T>(reinterpret_cast<const T*>(p.dy) + xrow0, (int64_t)H * P, P, PP, nv, nullptr, 0, dYT);
    stage<T>(reinterpret_cast<const T*>(p.x) + xrow0, (int64_t)H * P, P, PP, nv, nullptr, 0, XT);
    {
      const int t = lane;
      const bool valid = t < nv;
      float dtt, s_eff, cw[MP], ww[MP];
      token_controls<MP>(p, b, h, t0 + t, valid, lnt, dtt, s_eff, cw, ww);
      const float A = wave_inclusive_sum(dtt);
      const float Alast = uniform(__shfl(A, 63, 64));
      if (wave == 0) P_A[t] = A;
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        mode_scale(ms[m], rr[m], Alast);
        if ((m % NWT) != wave) continue;
        const float rho = expf(-dtt * rr[m]);
        const float kap = -expm1f(-dtt * rr[m]) * ww[m];
        const float ea = expf(-rr[m] * A);
        const float dec = expf(-rr[m] * (Alast - A)) * ms[m].E;
        P_O[m * kQ + t] = cw[m] * ea;
        P_Vt[m * kQ + t] = ms[m].safe ? kap * expf(rr[m] * A) : 0.0f;
        P_c[m * kQ + t] = cw[m];
        P_k[m * kQ + t] = kap;
        P_wdx[m * kQ + t] = kap * dec;
        P_wek[m * kQ + t] = rr[m] * kap * dec;
        P_wfk[m * kQ + t] = rr[m] * ww[m] * rho * dec;
        P_om[m * kQ + t] = cw[m] * ea * ms[m].upd;
      }
    }
    __syncthreads();

    // ---- adjoint-side terms: W_m = B G_m  ->  dx (inter), e / f (inter)
    floatx4 dxa[4];
    float ekf[16], fkf[16];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) dxa[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 16; ++j) ekf[j] = fkf[j] = 0.0f;
    if (active) {
      Frag<T> Bf[4][KBW];
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          const int n0 = nh * NBW * 16 + kb * 32;
          const T* row = Bs + (tb * 16 + li) * LDN + n0 + lg * 4;
          Bf[tb][kb] = frag_load4x2(row, (2 * kb + 1 < NBW) ? row + 16 : nullptr);
        }
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (m >= M) continue;
        Frag<T> Gf[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Gf[kb], s, Gs[m][2 * kb][s]);
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Gf[kb], 4 + s, (2 * kb + 1 < NBW) ? Gs[m][2 * kb + 1][s] : 0.0f);
        }
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
          floatx4 W = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) mma(W, Bf[tb][kb], Gf[kb]);
          const float4 wx = *reinterpret_cast<const float4*>(P_wdx + m * kQ + tb * 16 + lg * 4);
          const float4 we = *reinterpret_cast<const float4*>(P_wek + m * kQ + tb * 16 + lg * 4);
          const float4 wf = *reinterpret_cast<const float4*>(P_wfk + m * kQ + tb * 16 + lg * 4);
          dxa[tb][0] += wx.x * W[0];
          dxa[tb][1] += wx.y * W[1];
          dxa[tb][2] += wx.z * W[2];
          dxa[tb][3] += wx.w * W[3];
          ekf[tb * 4 + 0] += we.x * W[0];
          ekf[tb * 4 + 1] += we.y * W[1];
          ekf[tb * 4 + 2] += we.z * W[2];
          ekf[tb * 4 + 3] += we.w * W[3];
          fkf[tb * 4 + 0] += wf.x * W[0];
          fkf[tb * 4 + 1] += wf.y * W[1];
          fkf[tb * 4 + 2] += wf.z * W[2];
          fkf[tb * 4 + 3] += wf.w * W[3];
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float xv = to_f32(XT[pc * LDQ + tb * 16 + lg * 4 + r]);
          ekf[tb * 4 + r] *= xv;
          fkf[tb * 4 + r] *= xv;
        }
      if (NH > 1) {
        float* dst = YX + ((pb * 2 + nh) * 2) * 4 * 64;
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int tb = (1 - nh) * 2 + jj;
#pragma unroll
          for (int r = 0; r < 4; ++r) dst[(jj * 4 + r) * 64 + lane] = dxa[tb][r];
        }
      }
    }
    {
      const float ve = transpose_reduce16(ekf, li);
      const float vf = transpose_reduce16(fkf, li);
      redE[wave * kQ + tok_of(li, lg)] = ve;
      redF[wave * kQ + tok_of(li, lg)] = vf;
    }
    // ---- ((C B^T) o Gamma)^T tiles
    {
      const T* gt = gtiles + (((int64_t)b * nchunks + c) * p.G + g) * (kTiles * kTileElems);
      for (int tile = wave; tile < kTiles; tile += NWT) {
        const int tb = kTB[tile], kb = kKB[tile];
        float Gt[4];
        load_gtile(gt, tile, lane, Gt);
        floatx4 Gm = rank_m_tile<MP>(P_O, P_Vt, tb * 16, kb * 16, li, lg);
#pragma unroll
        for (int m = 0; m < MP; ++m) {
          if (ms[m].safe || m >= M) continue;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
            if (t >= k) Gm[r] += P_c[m * kQ + t] * P_k[m * kQ + k] * expf(-rr[m] * (P_A[t] - P_A[k]));
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
          GGT[k * LDQ + t] = (T)((t >= k) ? Gt[r] * Gm[r] : 0.0f);
        }
      }
    }

    __syncthreads();  // GGT, YX and the partials are complete

    if (wave == 0) {
      const int t = lane;
      float e = 0.f, f = 0.f;
      for (int w2 = 0; w2 < NWT; ++w2) {
        e += redE[w2 * kQ + t];
        f += redF[w2 * kQ + t];
      }
      if (t < nv) {
        const int64_t ith = ((int64_t)b * L + t0 + t) * H + h;
        eB[ith] = e;
        fB[ith] = f;
      }
    }

    if (active) {
      // ---- dx rows finished by this wave: other half + intra ((C B^T) o Gamma)^T dY + D dy
      T* dx = reinterpret_cast<T*>(p.dx);
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        if (NH > 1 && (tb >> 1) != nh) continue;
        if (NH > 1) {
          const float* src = YX + ((pb * 2 + (1 - nh)) * 2) * 4 * 64;
#pragma unroll
          for (int r = 0; r < 4; ++r) dxa[tb][r] += src[((tb & 1) * 4 + r) * 64 + lane];
        }
#pragma unroll
        for (int kk = tb / 2; kk < 2; ++kk) {
          const Frag<T> a = frag_load8(GGT + (tb * 16 + li) * LDQ + kk * 32 + lg * 8);
          const Frag<T> bb = frag_load8(dYT + pc * LDQ + kk * 32 + lg * 8);
          mma(dxa[tb], a, bb);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r;
          if (t < nv && pc < P) {
            const float dyv = to_f32(dYT[pc * LDQ + t]);
            dx[(((int64_t)b * L + t0 + t) * H + h) * P + pc] = (T)(dxa[tb][r] + Dh * dyv);
          }
        }
      }

      // ---- adjoint update G += C^T (omega o dY), rows n, columns p
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (!ms[m].ren) continue;
#pragma unroll
        for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
          for (int r = 0; r < 4; ++r) Gs[m][jb][r] *= ms[m].Enew;
      }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        float y8[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) y8[s] = to_f32(dYT[pc * LDQ + kt * 32 + lg * 8 + s]);
        Frag<T> Yf[MP];
#pragma unroll
        for (int m = 0; m < MP; ++m) {
          const float4 v0 = *reinterpret_cast<const float4*>(P_om + m * kQ + kt * 32 + lg * 8);
          const float4 v1 = *reinterpret_cast<const float4*>(P_om + m * kQ + kt * 32 + lg * 8 + 4);
          frag_set(Yf[m], 0, y8[0] * v0.x);
          frag_set(Yf[m], 1, y8[1] * v0.y);
          frag_set(Yf[m], 2, y8[2] * v0.z);
          frag_set(Yf[m], 3, y8[3] * v0.w);
          frag_set(Yf[m], 4, y8[4] * v1.x);
          frag_set(Yf[m], 5, y8[5] * v1.y);
          frag_set(Yf[m], 6, y8[6] * v1.z);
          frag_set(Yf[m], 7, y8[7] * v1.w);
        }
#pragma unroll
        for (int jb = 0; jb < NBW; ++jb) {
          const Frag<T> a = frag_load8(CT + ((nh * NBW + jb) * 16 + li) * LDQ + kt * 32 + lg * 8);
#pragma unroll
          for (int m = 0; m < MP; ++m)
            if (m < M) mma(Gs[m][jb], a, Yf[m]);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < MP; ++m) mode_scale_advance(ms[m]);
  }
}

// --------------------------------------------------------------------------
// sweep 2: reverse direction, adjoint transposed (rows p, columns n): dB

template <typename T, int MP, int NB>
__device__ __forceinline__ void sweep_adj_cols(const ScanParams& p, int b, int h, int g, T* __restrict__ dBp, unsigned char* smem) {
  constexpr int NP = NB * 16;
  const int PP = p.PP, PB = PP / 16, KP = (PB + 1) / 2;
  const int NWT = blockDim.x >> 6;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const bool active = wave < NB;
  const int ncol = wave * 16 + li;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M;
  const int nchunks = (L + kQ - 1) / kQ;

  T* Xs = reinterpret_cast<T*>(smem);  // [Q][LDP]
  T* dYs = Xs + kQ * LDP;              // [Q][LDP]
  T* dYT = dYs + kQ * LDP;             // [64][LDQ]
  T* CT = dYT + 64 * LDQ;              // [NP][LDQ]
  T* HGT = CT + NP * LDQ;              // [Q][LDQ]  (Gamma o dY X^T)^T
  float* P_O = reinterpret_cast<float*>(HGT + kQ * LDQ);
  float* P_Vt = P_O + MP * kQ;
  float* P_c = P_Vt + MP * kQ;
  float* P_k = P_c + MP * kQ;
  float* P_wdb = P_k + MP * kQ;  // kappa e^{-r(A_Q - A)} E
  float* P_om = P_wdb + MP * kQ; // c e^{-rA} * upd
  float* P_A = P_om + MP * kQ;

  float rr[MP], lnt[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    const float tau = (m < M) ? p.tau[m] : 1.0f;
    rr[m] = (m < M) ? 1.0f / tau : 0.0f;
    lnt[m] = (m < M) ? logf(tau) : 0.0f;
  }
  for (int i = tid; i < kQ * LDQ; i += blockDim.x) HGT[i] = (T)0.0f;

  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)M * N * P;
  floatx4 Gs[MP][kPBM];
  ModeScale ms[MP];
  {
    int lo = ncol * P + lg * 4;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      ms[m].E = 1.0f;
#pragma unroll
      for (int pb = 0; pb < kPBM; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pr = pb * 16 + lg * 4 + r;
          float v = 0.0f;
          if (p.d_final_state && active && m < M && ncol < N && pr < P)
            v = p.d_final_state[sbase + (int64_t)m * N * P + lo + pb * 16 + r];
          Gs[m][pb][r] = v;
        }
    }
  }

  for (int c = nchunks - 1; c >= 0; --c) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    __syncthreads();
    const int64_t xrow0 = (((int64_t)b * L + t0) * H + h) * P;
    const int64_t brow0 = (((int64_t)b * L + t0) * p.G + g) * N;
    stage<T>(reinterpret_cast<const T*>(p.x) + xrow0, (int64_t)H * P, P, PP, nv, Xs, LDP, nullptr);
    stage<T>(reinterpret_cast<const T*>(p.dy) + xrow0, (int64_t)H * P, P, PP, nv, dYs, LDP, dYT);
    stage<T>(reinterpret_cast<const T*>(p.Cm) + brow0, (int64_t)p.G * N, N, NP, nv, nullptr, 0, CT);
    {
      const int t = lane;
      const bool valid = t < nv;
      float dtt, s_eff, cw[MP], ww[MP];
      token_controls<MP>(p, b, h, t0 + t, valid, lnt, dtt, s_eff, cw, ww);
      const float A = wave_inclusive_sum(dtt);
      const float Alast = uniform(__shfl(A, 63, 64));
      if (wave == 0) P_A[t] = A;
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        mode_scale(ms[m], rr[m], Alast);
        if ((m % NWT) != wave) continue;
        const float kap = -expm1f(-dtt * rr[m]) * ww[m];
        const float ea = expf(-rr[m] * A);
        P_O[m * kQ + t] = cw[m] * ea;
        P_Vt[m * kQ + t] = ms[m].safe ? kap * expf(rr[m] * A) : 0.0f;
        P_c[m * kQ + t] = cw[m];
        P_k[m * kQ + t] = kap;
        P_wdb[m * kQ + t] = kap * expf(-rr[m] * (Alast - A)) * ms[m].E;
        P_om[m * kQ + t] = cw[m] * ea * ms[m].upd;
      }
    }
    __syncthreads();

    // ---- V_m = X G_m^T  ->  dB (inter)
    floatx4 dBa[4];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) dBa[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (active) {
      Frag<T> Af[4][2];
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int kp = 0; kp < 2; ++kp) {
          Af[tb][kp] = frag_zero<T>();
          if (kp < KP) {
            const T* row = Xs + (tb * 16 + li) * LDP + kp * 32 + lg * 4;
            Af[tb][kp] = frag_load4x2(row, (2 * kp + 1 < PB) ? row + 16 : nullptr);
          }
        }
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (m >= M) continue;
        Frag<T> Gf[2];
#pragma unroll
        for (int kp = 0; kp < 2; ++kp) {
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Gf[kp], s, Gs[m][2 * kp][s]);
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Gf[kp], 4 + s, Gs[m][2 * kp + 1][s]);
        }
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
          floatx4 V = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kp = 0; kp < 2; ++kp)
            if (kp < KP) mma(V, Af[tb][kp], Gf[kp]);
          const float4 wb = *reinterpret_cast<const float4*>(P_wdb + m * kQ + tb * 16 + lg * 4);
          dBa[tb][0] += wb.x * V[0];
          dBa[tb][1] += wb.y * V[1];
          dBa[tb][2] += wb.z * V[2];
          dBa[tb][3] += wb.w * V[3];
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // ---- (Gamma o dY X^T)^T tiles
    for (int tile = wave; tile < kTiles; tile += NWT) {
      const int tb = kTB[tile], kb = kKB[tile];
      const floatx4 D = dyx_tile<T>(dYs, Xs, tb, kb, PP, li, lg);
      floatx4 Gm = rank_m_tile<MP>(P_O, P_Vt, tb * 16, kb * 16, li, lg);
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (ms[m].safe || m >= M) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
          if (t >= k) Gm[r] += P_c[m * kQ + t] * P_k[m * kQ + k] * expf(-rr[m] * (P_A[t] - P_A[k]));
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
        HGT[k * LDQ + t] = (T)((t >= k) ? Gm[r] * D[r] : 0.0f);
      }
    }

    __syncthreads();  // HGT complete

    if (active) {
      // ---- dB intra: (Gamma o dY X^T)^T C, rows k, contraction over t >= k
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int kk = tb / 2; kk < 2; ++kk) {
          const Frag<T> a = frag_load8(HGT + (tb * 16 + li) * LDQ + kk * 32 + lg * 8);
          const Frag<T> bb = frag_load8(CT + ncol * LDQ + kk * 32 + lg * 8);
          mma(dBa[tb], a, bb);
        }
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r;
          if (t < nv && ncol < N) dBp[(((int64_t)b * L + t0 + t) * H + h) * N + ncol] = (T)dBa[tb][r];
        }

      // ---- adjoint update G^T += dY^T (omega o C), rows p, columns n
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (!ms[m].ren) continue;
#pragma unroll
        for (int pb = 0; pb < kPBM; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r) Gs[m][pb][r] *= ms[m].Enew;
      }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        float c8[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) c8[s] = to_f32(CT[ncol * LDQ + kt * 32 + lg * 8 + s]);
        Frag<T> Cf[MP];
#pragma unroll
        for (int m = 0; m < MP; ++m) {
          const float4 v0 = *reinterpret_cast<const float4*>(P_om + m * kQ + kt * 32 + lg * 8);
          const float4 v1 = *reinterpret_cast<const float4*>(P_om + m * kQ + kt * 32 + lg * 8 + 4);
          frag_set(Cf[m], 0, c8[0] * v0.x);
          frag_set(Cf[m], 1, c8[1] * v0.y);
          frag_set(Cf[m], 2, c8[2] * v0.z);
          frag_set(Cf[m], 3, c8[3] * v0.w);
          frag_set(Cf[m], 4, c8[4] * v1.x);
          frag_set(Cf[m], 5, c8[5] * v1.y);
          frag_set(Cf[m], 6, c8[6] * v1.z);
          frag_set(Cf[m], 7, c8[7] * v1.w);
        }
#pragma unroll
        for (int pb = 0; pb < kPBM; ++pb) {
          if (pb >= PB) continue;
          const Frag<T> a = frag_load8(dYT + (pb * 16 + li) * LDQ + kt * 32 + lg * 8);
#pragma unroll
          for (int m = 0; m < MP; ++m)
            if (m < M) mma(Gs[m][pb], a, Cf[m]);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < MP; ++m) mode_scale_advance(ms[m]);
  }
}

// --------------------------------------------------------------------------

struct BwdWork {
  void* tiles;
  void* dBp;
  void* dCp;
  float* eA;
  float* fA;
  float* eB;
  float* fB;
  float* F;
  float* dDp;
};

template <typename T, int MP, int NB>
__global__ void __launch_bounds__(512) frac_bwd_kernel(ScanParams p, BwdWork wk) {
  extern __shared__ __align__(16) unsigned char smem[];
  // XCD-aware (batch, head) order as in the forward
  int j = blockIdx.x;
  const int nblk = gridDim.x;
  if ((nblk & 7) == 0) j = (blockIdx.x & 7) * (nblk >> 3) + (blockIdx.x >> 3);
  const int b = j / p.H, h = j - b * p.H, g = h * p.G / p.H;
  const T* tiles = reinterpret_cast<const T*>(wk.tiles);
  if (blockIdx.y == 0)
    sweep_state<T, MP, NB>(p, b, h, g, tiles, reinterpret_cast<T*>(wk.dCp), wk.eA, wk.fA, wk.F, wk.dDp, smem);
  else if (blockIdx.y == 1)
    sweep_adj_rows<T, MP, NB>(p, b, h, g, tiles, wk.eB, wk.fB, smem);
  else
    sweep_adj_cols<T, MP, NB>(p, b, h, g, reinterpret_cast<T*>(wk.dBp), smem);
}

template <typename T, int MP, int NB>
size_t bwd_lds_bytes(int PP) {
  constexpr int NP = NB * 16;
  const size_t s0 = sizeof(T) * (size_t)(kQ * LDP + 64 * LDQ + kQ * LDP + 2 * NP * LDQ + kQ * LDQ) +
                    sizeof(float) * (size_t)(10 * MP * kQ + kQ + 2 * 8 * kQ + 3 * kTiles * 16);
  const size_t s1 = sizeof(T) * (size_t)(kQ * (NP + 8) + NP * LDQ + 2 * 64 * LDQ + kQ * LDQ) +
                    sizeof(float) * (size_t)(8 * MP * kQ + kQ + 4 * 1024 + 2 * 8 * kQ);
  const size_t s2 = sizeof(T) * (size_t)(2 * kQ * LDP + 64 * LDQ + NP * LDQ + kQ * LDQ) +
                    sizeof(float) * (size_t)(6 * MP * kQ + kQ);
  (void)PP;
  return s0 > s1 ? (s0 > s2 ? s0 : s2) : (s1 > s2 ? s1 : s2);
}

// ddt from the per-token terms: suffix sums over the sequence, one wave per (batch, head).
__global__ void __launch_bounds__(64) frac_bwd_ddt_kernel(ScanParams p, const float* __restrict__ eA,
                                                         const float* __restrict__ fA, const float* __restrict__ eB,
                                                         const float* __restrict__ fB, const float* __restrict__ F,
                                                         const float* __restrict__ dDp) {
  const int bh = blockIdx.x, b = bh / p.H, h = bh - b * p.H;
  const int lane = threadIdx.x;
  const int L = p.L, H = p.H;
  float carry = 0.0f;  // sum of e over the tokens after the current chunk
  const float Fv = F[bh];
  for (int c = (L + kQ - 1) / kQ - 1; c >= 0; --c) {
    const int t0 = c * kQ, t = t0 + lane;
    const bool valid = t < L;
    const int64_t ith = ((int64_t)b * L + t) * H + h;
    const float e = valid ? eA[ith] - eB[ith] : 0.0f;
    // inclusive suffix sum within the chunk (lane order reversed)
    float s = e;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float o = __shfl_down(s, off, 64);
      if (lane + off < 64) s += o;
    }
    if (valid) {
      const float al = strided3(p.alpha, p.as0, p.as1, p.as2, b, t, h);
      const float lam = p.lambda ? strided3(p.lambda, p.ls0, p.ls1, p.ls2, b, t, h) : 1.0f;
      const float s_eff = p.lambda ? exp2f(log2f(lam) / al) : 1.0f;
      const float ddtt = -Fv - (carry + s) + fA[ith] + fB[ith];
      p.ddt[ith] = ddtt * s_eff;
    }
    carry += __shfl(s, 0, 64);
  }
  if (p.dD && b == 0 && lane == 0) {
    float acc = 0.0f;
    for (int bb = 0; bb < p.Bsz; ++bb) acc += dDp[(int64_t)bb * H + h];
    p.dD[h] = acc;
  }
}

// dB, dC of each group: fixed-order sum of the per-head partials.
template <typename T>
__global__ void __launch_bounds__(128) frac_bwd_group_sum_kernel(ScanParams p, const T* __restrict__ dBp,
                                                                 const T* __restrict__ dCp) {
  const int64_t bt = blockIdx.x;  // b * L + t
  const int g = blockIdx.y;
  const int H = p.H, N = p.N, hpg = H / p.G;
  T* dB = reinterpret_cast<T*>(p.dBm);
  T* dC = reinterpret_cast<T*>(p.dCm);
  for (int n = threadIdx.x; n < N; n += blockDim.x) {
    float sb = 0.f, sc = 0.f;
    for (int j = 0; j < hpg; ++j) {
      const int64_t off = (bt * H + g * hpg + j) * N + n;
      sb += to_f32(dBp[off]);
      sc += to_f32(dCp[off]);
    }
    const int64_t o = (bt * p.G + g) * N + n;
    dB[o] = (T)sb;
    dC[o] = (T)sc;
  }
}

struct BwdLayout {
  size_t tiles, dBp, dCp, scal, total;
};

BwdLayout bwd_layout(const ScanParams& p) {
  BwdLayout l{};
  const size_t es = p.io_bf16 ? 2 : 4;
  const size_t bl = (size_t)p.Bsz * p.L;
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  l.tiles = 0;
  l.dBp = up(cb_tiles_bytes(p));
  l.dCp = l.dBp + up(bl * p.H * p.N * es);
  l.scal = l.dCp + up(bl * p.H * p.N * es);
  l.total = l.scal + up(sizeof(float) * (4 * bl * p.H + 2 * (size_t)p.Bsz * p.H));
  return l;
}

template <typename T, int MP, int NB>
hipError_t launch_bwd_variant(const ScanParams& p, void* ws, hipStream_t stream) {
  const BwdLayout l = bwd_layout(p);
  unsigned char* base = reinterpret_cast<unsigned char*>(ws);
  BwdWork wk;
  wk.tiles = base + l.tiles;
  wk.dBp = base + l.dBp;
  wk.dCp = base + l.dCp;
  float* sc = reinterpret_cast<float*>(base + l.scal);
  const size_t blh = (size_t)p.Bsz * p.L * p.H;
  wk.eA = sc;
  wk.fA = sc + blh;
  wk.eB = sc + 2 * blh;
  wk.fB = sc + 3 * blh;
  wk.F = sc + 4 * blh;
  wk.dDp = wk.F + (size_t)p.Bsz * p.H;

  hipError_t e = launch_cb_tiles(p, wk.tiles, stream);
  if (e != hipSuccess) return e;
  const int nw_state = NB, nw_rows = (p.PP / 16) * (NB >= 2 ? 2 : 1);
  const int nwt = nw_state > nw_rows ? nw_state : nw_rows;
  const size_t lds = bwd_lds_bytes<T, MP, NB>(p.PP);
  auto kern = frac_bwd_kernel<T, MP, NB>;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(p.Bsz * p.H, 3), dim3(64 * nwt), lds, stream, p, wk);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(frac_bwd_ddt_kernel, dim3(p.Bsz * p.H), dim3(64), 0, stream, p, wk.eA, wk.fA, wk.eB, wk.fB,
                     wk.F, wk.dDp);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((frac_bwd_group_sum_kernel<T>), dim3((unsigned)(p.Bsz * p.L), p.G), dim3(128), 0, stream, p,
                     reinterpret_cast<const T*>(wk.dBp), reinterpret_cast<const T*>(wk.dCp));
  return hipGetLastError();
}

template <typename T, int MP>
hipError_t launch_bwd_nb(const ScanParams& p, void* ws, hipStream_t stream) {
  switch (p.NP / 16) {
    case 1: return launch_bwd_variant<T, MP, 1>(p, ws, stream);
    case 2: return launch_bwd_variant<T, MP, 2>(p, ws, stream);
    case 4: return launch_bwd_variant<T, MP, 4>(p, ws, stream);
    case 8: return launch_bwd_variant<T, MP, 8>(p, ws, stream);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch_bwd_mp(const ScanParams& p, void* ws, hipStream_t stream) {
  if (p.M <= 1) return launch_bwd_nb<T, 1>(p, ws, stream);
  if (p.M <= 2) return launch_bwd_nb<T, 2>(p, ws, stream);
  if (p.M <= 4) return launch_bwd_nb<T, 4>(p, ws, stream);
  return launch_bwd_nb<T, 8>(p, ws, stream);
}

}  // namespace

size_t scan_bwd_workspace(const ScanParams& p) {
  if (p.Bsz == 0 || p.L == 0) return 0;
  return bwd_layout(p).total;
}

hipError_t launch_scan_bwd(const ScanParams& p, void* ws, size_t, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  return p.io_bf16 ? launch_bwd_mp<bf16>(p, ws, stream) : launch_bwd_mp<float>(p, ws, stream);
}

}  // namespace frac
