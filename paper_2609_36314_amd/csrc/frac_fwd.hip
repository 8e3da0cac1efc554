// frac_fwd.hip -- chunked parallel scan, forward (prefill / training forward).
//
// Method: the selective mode-bank recurrence of Sec. 3.2 (eq. frac-selective-update,
// eq. frac-readout) with a B/C-widened N x P state per mode, evaluated chunk by
// chunk as in the remark closing Sec. 3.2 and the appendix on the efficient
// implementation.  Inside a chunk of Q tokens, with A_t the chunk-local inclusive
// sum of the effective steps dtt and r_m = 1 / tau_m:
//
//   y_t = sum_m c_{t,m} e^{-r_m A_t} C_t^T S_m            (state entering the chunk)
//       + sum_{k<=t} (C_t . B_k) Gamma_{t,k} x_k            (intra-chunk mixing)
//       + D x_t
//   Gamma_{t,k} = sum_m c_{t,m} kappa_{k,m} e^{-r_m (A_t - A_k)}
//   S_m <- e^{-r_m A_Q} S_m + sum_k kappa_{k,m} e^{-r_m (A_Q - A_k)} B_k x_k^T
//
// The decay between two tokens is always formed from a difference of chunk-local
// cumulative steps (the log-space form of the appendix), never from a ratio of
// sequence-global products.
//
// Kernels:
//   frac_cb_kernel   G_chunk = C B^T (Q x Q, causal 16x16 tiles) once per
//                    (batch, chunk, group) -- shared by every head of the group --
//                    stored in the per-lane fragment order the scan reads back.
//   frac_fwd_kernel  one workgroup per (batch, head).  Wave (pb, nh) owns state
//                    columns p in [16 pb, 16 pb + 16) and, when N >= 32, one half
//                    of the N rows, for every mode.  Its share of the float32
//                    M x N x P state lives in matrix-core accumulator registers
//                    for the whole sequence and never touches memory.  Per chunk:
//                    stage x (transposed), B (transposed) and C in LDS; per-token
//                    controls and weights (lane = token); (G o Gamma) tiles split
//                    over the waves; readout, intra-chunk product and state update
//                    as 16x16x32 matrix-core products (bfloat16 operands, float32
//                    accumulation).  The accumulator tiles of the state are
//                    converted in registers straight into B operands of the
//                    readout: their row order becomes the K-slot order, matched by
//                    the order in which C is read from LDS.
//
// Gamma uses the factorised form (c e^{-r A_t}) (kappa e^{r A_k}) through a float32
// 16x16x4 product with the modes as K, for every mode whose chunk decay r_m A_Q
// stays below 55 (so e^{r A_k} cannot overflow); other modes fall back to one exp
// per (t, k) pair.  The per-mode decay of the state is not applied to the
// accumulators every chunk: the state is held as E_m * S^_m with a float scale E_m
// that absorbs the chunk decays, and the accumulators are rescaled only when E_m
// would fall below 2^-60.
#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

// lower-triangular 16x16 tiles of the Q x Q matrix: (row block, column block)
__constant__ int kTileTB[10] = {0, 1, 1, 2, 2, 2, 3, 3, 3, 3};
__constant__ int kTileKB[10] = {0, 0, 1, 0, 1, 2, 0, 1, 2, 3};
constexpr int kTiles = 10;
constexpr int kTileElems = 256;  // one 16x16 tile: 64 lanes x 4 values

constexpr float kSafeExponent = 55.0f;  // e^{r A} <= e^55 ~ 7.7e23
constexpr float kRescaleFloor = 0x1p-60f;

// Broadcast lane 0's value as a wave-uniform scalar.  The builtin moves 32-bit
// integers, so the float travels as its bit pattern.
__device__ __forceinline__ float uniform(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

// --------------------------------------------------------------- C B^T tiles

template <typename T, int NB>
__global__ void __launch_bounds__(256) frac_cb_kernel(ScanParams p, T* __restrict__ gtiles) {
  constexpr int NP = NB * 16;
  constexpr int LDN = NP + 8;
  constexpr int KB = (NB + 1) / 2;
  const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int nchunks = gridDim.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, N = p.N, G = p.G;
  const int t0 = c * kQ, nv = min(kQ, L - t0);

  extern __shared__ __align__(16) unsigned char smem[];
  T* Cs = reinterpret_cast<T*>(smem);
  T* Bs = Cs + kQ * LDN;
  const T* Bg = reinterpret_cast<const T*>(p.Bm);
  const T* Cg = reinterpret_cast<const T*>(p.Cm);
  constexpr int ngroups = NP / 8;
  for (int idx = tid; idx < kQ * ngroups; idx += 256) {
    const int t = idx / ngroups, n0 = (idx - t * ngroups) * 8;
    if (t < nv && n0 < N) {
      const int64_t off = (((int64_t)b * L + t0 + t) * G + g) * N + n0;
      copy8(Cs + t * LDN + n0, Cg + off);
      copy8(Bs + t * LDN + n0, Bg + off);
    } else {
      zero8(Cs + t * LDN + n0);
      zero8(Bs + t * LDN + n0);
    }
  }
  __syncthreads();
  T* out = gtiles + (((int64_t)b * nchunks + c) * G + g) * (kTiles * kTileElems);
  for (int tile = wave; tile < kTiles; tile += 4) {
    const int tb = kTileTB[tile], kb = kTileKB[tile];
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      const int n0 = kk * 32 + lg * 8;
      Frag<T> a = frag_zero<T>(), bb = frag_zero<T>();
      if (n0 < NP) {
        a = frag_load8(Cs + (tb * 16 + li) * LDN + n0);
        bb = frag_load8(Bs + (kb * 16 + li) * LDN + n0);
      }
      mma(acc, a, bb);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) out[tile * kTileElems + lane * 4 + r] = (T)acc[r];
  }
}

// ------------------------------------------------------------------- the scan

// LDS row strides (elements) of the staged tiles; padded so that the transposed
// fragment reads of 4 consecutive rows and the row reads of 16 rows spread over
// the LDS banks.  bfloat16 tiles are double-buffered: the next chunk is copied
// in (direct global -> LDS) while the current one is computed.
template <typename T, int NB>
struct FwdCfg {
  static constexpr int NP = NB * 16;
  static constexpr bool kBf16 = sizeof(T) == 2;
  static constexpr int XS = kBf16 ? 64 + 8 : 64 + 4;    // x tile   [t][p]
  static constexpr int BS = kBf16 ? NP + 16 : NP + 8;   // B tile   [t][n]
  static constexpr int CS = kBf16 ? NP + 8 : NP + 4;    // C tile   [t][n]
  static constexpr int GS = kBf16 ? 64 + 8 : 64 + 4;    // ((C B^T) o Gamma)^T [k][t]
  static constexpr int NBUF = kBf16 ? 2 : 1;
};

template <typename T, int MP, int NB>
__global__ void __launch_bounds__(512) frac_fwd_kernel(ScanParams p, const T* __restrict__ gtiles) {
  using Cfg = FwdCfg<T, NB>;
  constexpr int NP = Cfg::NP, XS = Cfg::XS, BS = Cfg::BS, CS = Cfg::CS, GS = Cfg::GS;
  constexpr int NH = NB >= 2 ? 2 : 1;     // N halves (waves per p-block)
  constexpr int NBW = NB / NH;            // 16-row blocks of N owned by a wave
  constexpr int KBW = (NBW + 1) / 2;      // 32-row K steps of the readout per wave
  const int NWT = blockDim.x >> 6;        // waves in the workgroup
  const int NW = NWT / NH;                // p-blocks
  const int PP = NW * 16;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int pb = wave % NW, nh = wave / NW;
  const int pc = pb * 16 + li;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M, G = p.G;
  const int nchunks = (L + kQ - 1) / kQ;

  // Blocks are dealt round-robin to the 8 XCDs; give each XCD a contiguous run of
  // (batch, head) so that heads sharing B and C share one L2.
  int j = blockIdx.x;
  const int nblk = gridDim.x;
  if ((nblk & 7) == 0) j = (blockIdx.x & 7) * (nblk >> 3) + (blockIdx.x >> 3);
  const int b = j / H, h = j - b * H, g = h * G / H;

  __shared__ __align__(16) T Xb0[64 * XS], Bb0[64 * BS], Cb0[64 * CS];
  __shared__ __align__(16) T Xb1[Cfg::NBUF == 2 ? 64 * XS : 8], Bb1[Cfg::NBUF == 2 ? 64 * BS : 8],
      Cb1[Cfg::NBUF == 2 ? 64 * CS : 8];
  __shared__ __align__(16) T GGT[64 * GS];   // ((C B^T) o Gamma)^T of the chunk, causal
  __shared__ __align__(16) T Yb[64 * XS];    // output rows of the previous chunk
  __shared__ __align__(16) float prm[6 * MP * kQ + kQ];
  __shared__ __align__(16) float YX[NH > 1 ? 4 * 1024 : 4];
  float* P_om = prm;              // [MP][Q] c e^{-rA_t} E_m        (readout)
  float* P_v = P_om + MP * kQ;    // [MP][Q] kappa e^{-r(A_Q-A_t)} upd (update)
  float* P_O = P_v + MP * kQ;     // [MP][Q] c e^{-r A_t}            (Gamma rows)
  float* P_Vt = P_O + MP * kQ;    // [MP][Q] kappa e^{r A_t}, safe modes (Gamma columns)
  float* P_c = P_Vt + MP * kQ;    // [MP][Q] c      (modes past the factorisation bound)
  float* P_k = P_c + MP * kQ;     // [MP][Q] kappa
  float* P_A = P_k + MP * kQ;     // [Q] A_t

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * P;
  const T* Bgp = reinterpret_cast<const T*>(p.Bm) + (((int64_t)b * L) * G + g) * N;
  const T* Cgp = reinterpret_cast<const T*>(p.Cm) + (((int64_t)b * L) * G + g) * N;
  T* yg = reinterpret_cast<T*>(p.y) + (((int64_t)b * L) * H + h) * P;
  const int64_t xstride = (int64_t)H * P, bstride = (int64_t)G * N;

  // per-mode rates 1/tau_m and log tau_m, read from LDS where needed
  __shared__ float s_rr[MP], s_lnt[MP];
  if (tid < MP) {
    const float tau = (tid < M) ? p.tau[tid] : 1.0f;
    s_rr[tid] = (tid < M) ? 1.0f / tau : 0.0f;
    s_lnt[tid] = (tid < M) ? logf(tau) : 0.0f;
  }
  for (int i = tid; i < 64 * GS; i += blockDim.x) GGT[i] = (T)0.0f;

  // ---- state: S[m][jb] holds rows n = 16 (nh NBW + jb) + 4 lg + r, column pc
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)M * N * P;
  floatx4 S[MP][NBW];
  float E[MP];
  {
    // lane offset kept opaque so that the final store cannot share (and keep alive
    // across the sequence loop) the per-element offsets of this load
    int lo = (nh * NBW * 16 + lg * 4) * P + pc;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      E[m] = 1.0f;
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = (nh * NBW + jb) * 16 + lg * 4 + r;
          float v = 0.0f;
          if (p.init_state && m < M && n < N && pc < P)
            v = p.init_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * P];
          S[m][jb][r] = v;
        }
    }
  }
  const float Dh = p.D ? p.D[h] : 0.0f;
  const bool w_is_c = p.write_logit == p.read_logit;  // then the write weights equal the read weights

  // per-token controls of a chunk, loaded one chunk ahead (lane = token)
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const int64_t al_st = p.as1;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const int64_t lm_st = p.ls1;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const int64_t lg_st = (int64_t)H * M;
  auto load_controls = [&](int c, float& dtv, float& al, float& lam) {
    const int tg = c * kQ + lane;
    const bool valid = tg < L;
    dtv = valid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al = valid ? al_bh[tg * al_st] : 1.0f;
    lam = (valid && lm_bh) ? lm_bh[tg * lm_st] : 1.0f;
  };
  auto stage = [&](int c, T* Xd, T* Bd, T* Cd) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    dma_tile<T>(Xd, xg + (int64_t)t0 * xstride, xstride, P, XS, nv);
    dma_tile<T>(Bd, Bgp + (int64_t)t0 * bstride, bstride, N, BS, nv);
    dma_tile<T>(Cd, Cgp + (int64_t)t0 * bstride, bstride, N, CS, nv);
  };
  // output rows of chunk c (staged in Yb) -> global, 16 bytes per thread
  auto store_y = [&](int c) {
    constexpr int E8 = 16 / sizeof(T);
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    const int cpr = P / E8;
    for (int i = tid; i < nv * cpr; i += blockDim.x) {
      const int t = i / cpr, ch = i - t * cpr;
      *reinterpret_cast<int4*>(yg + (int64_t)(t0 + t) * xstride + ch * E8) =
          *reinterpret_cast<const int4*>(Yb + t * XS + ch * E8);
    }
  };

  float dt_n, al_n, lam_n;
  load_controls(0, dt_n, al_n, lam_n);
  if (Cfg::NBUF == 2) stage(0, Xb0, Bb0, Cb0);

  // one chunk: Xc/Bc/Cc hold it (or receive it when single-buffered), Xn/Bn/Cn
  // receive the next one
  auto step = [&](int c, T* Xc, T* Bc, T* Cc, T* Xn, T* Bn, T* Cn) __attribute__((always_inline)) {
    const int t0 = c * kQ;
    const int nv = min(kQ, L - t0);
    wait_vmem();
    barrier();  // this chunk's tiles have landed; every wave is done with the previous chunk
    if (c > 0) store_y(c - 1);
    if (Cfg::NBUF == 2) {
      if (c + 1 < nchunks) stage(c + 1, Xn, Bn, Cn);
    } else {
      stage(c, Xc, Bc, Cc);
      wait_vmem();
      barrier();
    }
    const float dtv = dt_n, al = al_n, lam = lam_n;
    if (c + 1 < nchunks) load_controls(c + 1, dt_n, al_n, lam_n);

    // ---- controls and weights, lane = token; wave w stores modes m % NWT == w
    // per-mode flags as scalar bit masks: bit m of `renbits` set = the state of
    // mode m is folded back to unit scale after this chunk, bit m of `unsafe` set
    // = the factorised Gamma would overflow for mode m (direct decay instead)
    float renf[MP];
    int renbits = 0, unsafe = 0;
    {
      const int t = lane;
      const bool valid = t < nv;
      const int64_t ith = (int64_t)(t0 + t) * lg_st;
      const float s_eff = lm_bh ? exp2f(log2f(lam) / al) : 1.0f;
      const float dtt = valid ? dtv * s_eff : 0.0f;
      const float A = wave_inclusive_sum(dtt);
      const float Alast = uniform(__shfl(A, 63, 64));
      float zc[MP], zw[MP];
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        const float prior = -al * s_lnt[m];
        zc[m] = prior + ((rl_bh && valid && m < M) ? rl_bh[ith + m] : 0.0f);
        zw[m] = prior + ((wl_bh && valid && m < M) ? wl_bh[ith + m] : 0.0f);
      }
      softmax_fast<MP>(zc, M);
      if (w_is_c) {
#pragma unroll
        for (int m = 0; m < MP; ++m) zw[m] = zc[m];
      } else {
        softmax_fast<MP>(zw, M);
      }
      if (wave == 0) P_A[t] = A;
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        const float r = s_rr[m];
        // r A_Q and the new scale are wave-uniform and non-negative: compare bit patterns
        const float xr = uniform(r * Alast);
        const bool safe = __float_as_int(xr) <= __float_as_int(kSafeExponent);
        if (m < M && !safe) unsafe |= 1 << m;
        const float Enew = uniform(E[m] * fexp(-xr));
        const bool ren = __float_as_int(Enew) < __float_as_int(kRescaleFloor);
        if (ren) renbits |= 1 << m;
        renf[m] = Enew;
        if ((m % NWT) != wave) continue;
        const float upd = ren ? 1.0f : __frcp_rn(Enew);
        const float kap = one_minus_exp_neg(dtt * r) * zw[m];
        const float om = zc[m] * fexp(-r * A);
        P_O[m * kQ + t] = om;
        P_om[m * kQ + t] = om * E[m];
        P_v[m * kQ + t] = kap * fexp(-r * (Alast - A)) * upd;
        P_Vt[m * kQ + t] = safe ? kap * fexp(r * A) : 0.0f;
        P_c[m * kQ + t] = zc[m];
        P_k[m * kQ + t] = kap;
      }
    }
    barrier();  // controls in LDS

    // ---- ((C B^T) o Gamma)^T, lower-triangular 16x16 tiles split over the waves
    {
      const T* gt = gtiles + (((int64_t)b * nchunks + c) * G + g) * (kTiles * kTileElems);
      for (int tile = wave; tile < kTiles; tile += NWT) {
        const int tb = kTileTB[tile], kb = kTileKB[tile];
        float Gt[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) Gt[r] = to_f32(gt[tile * kTileElems + lane * 4 + r]);
        floatx4 Gm = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < (MP + 3) / 4; ++q) {
          const int m = q * 4 + lg;
          const float av = (m < MP) ? P_O[m * kQ + tb * 16 + li] : 0.0f;
          const float bv = (m < MP) ? P_Vt[m * kQ + kb * 16 + li] : 0.0f;
          Gm = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, Gm, 0, 0, 0);
        }
        if (unsafe) {
          for (int m = 0; m < MP; ++m) {
            if (!((unsafe >> m) & 1)) continue;
            const float rm = s_rr[m];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
              if (t >= k) Gm[r] += P_c[m * kQ + t] * P_k[m * kQ + k] * fexp(-rm * (P_A[t] - P_A[k]));
            }
          }
        }
        T* dst = GGT + (kb * 16 + li) * GS + tb * 16 + lg * 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
          dst[r] = (T)((t >= k) ? Gt[r] * Gm[r] : 0.0f);
        }
      }
    }

    // ---- readout of the state entering the chunk (this wave's rows of N)
    floatx4 Y[4];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) Y[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    {
      Frag<T> Ca[4][KBW];
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          const T* row = Cc + (tb * 16 + li) * CS + nh * NBW * 16 + kb * 32 + lg * 4;
          Ca[tb][kb] = frag_load4x2(row, (2 * kb + 1 < NBW) ? row + 16 : nullptr);
        }
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (m >= M) continue;
        Frag<T> Sf[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Sf[kb], s, S[m][2 * kb][s]);
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Sf[kb], 4 + s, (2 * kb + 1 < NBW) ? S[m][2 * kb + 1][s] : 0.0f);
        }
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
          floatx4 Z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) mma(Z, Ca[tb][kb], Sf[kb]);
          const float4 om = *reinterpret_cast<const float4*>(P_om + m * kQ + tb * 16 + lg * 4);
          Y[tb][0] += om.x * Z[0];
          Y[tb][1] += om.y * Z[1];
          Y[tb][2] += om.z * Z[2];
          Y[tb][3] += om.w * Z[3];
        }
      }
    }
    if (NH > 1) {
      // hand the row blocks finished by the other N half over through LDS
      float* dst = YX + ((pb * 2 + nh) * 2) * 4 * 64;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int tb = (1 - nh) * 2 + jj;
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[(jj * 4 + r) * 64 + lane] = Y[tb][r];
      }
    }
    barrier();  // GGT and YX complete

    // ---- intra-chunk product, skip term, output rows into Yb
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      if (NH > 1 && (tb >> 1) != nh) continue;
      if (NH > 1) {
        const float* src = YX + ((pb * 2 + (1 - nh)) * 2) * 4 * 64;
#pragma unroll
        for (int r = 0; r < 4; ++r) Y[tb][r] += src[((tb & 1) * 4 + r) * 64 + lane];
      }
#pragma unroll
      for (int kk = 0; kk <= tb / 2; ++kk) {
        const Frag<T> a = frag_load_rows(GGT, GS, kk * 32 + lg * 8, tb * 16);
        const Frag<T> bb = frag_load_rows(Xc, XS, kk * 32 + lg * 8, pb * 16);
        mma(Y[tb], a, bb);
      }
      float xv[4];
      col4_rows(Xc, XS, tb * 16 + lg * 4, pb * 16, xv);
#pragma unroll
      for (int r = 0; r < 4; ++r) Yb[(tb * 16 + lg * 4 + r) * XS + pc] = (T)(Y[tb][r] + Dh * xv[r]);
    }

    // ---- state update  S_m <- (rescale) + B^T (v_m o X)
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      if (!((renbits >> m) & 1)) continue;
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) S[m][jb][r] *= renf[m];
    }
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const Frag<T> xf = frag_load_rows(Xc, XS, kt * 32 + lg * 8, pb * 16);
      float xs[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) xs[s] = to_f32(xf.v[s]);
      Frag<T> a[NBW];
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb) a[jb] = frag_load_rows(Bc, BS, kt * 32 + lg * 8, (nh * NBW + jb) * 16);
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (m >= M) continue;
        const float4 v0 = *reinterpret_cast<const float4*>(P_v + m * kQ + kt * 32 + lg * 8);
        const float4 v1 = *reinterpret_cast<const float4*>(P_v + m * kQ + kt * 32 + lg * 8 + 4);
        Frag<T> Xf;
        frag_set(Xf, 0, xs[0] * v0.x);
        frag_set(Xf, 1, xs[1] * v0.y);
        frag_set(Xf, 2, xs[2] * v0.z);
        frag_set(Xf, 3, xs[3] * v0.w);
        frag_set(Xf, 4, xs[4] * v1.x);
        frag_set(Xf, 5, xs[5] * v1.y);
        frag_set(Xf, 6, xs[6] * v1.z);
        frag_set(Xf, 7, xs[7] * v1.w);
#pragma unroll
        for (int jb = 0; jb < NBW; ++jb) mma(S[m][jb], a[jb], Xf);
      }
    }
#pragma unroll
    for (int m = 0; m < MP; ++m) E[m] = ((renbits >> m) & 1) ? 1.0f : renf[m];
  };

  for (int c = 0; c < nchunks; c += 2) {
    step(c, Xb0, Bb0, Cb0, Xb1, Bb1, Cb1);
    if (c + 1 < nchunks) {
      if (Cfg::NBUF == 2) step(c + 1, Xb1, Bb1, Cb1, Xb0, Bb0, Cb0);
      else step(c + 1, Xb0, Bb0, Cb0, Xb0, Bb0, Cb0);
    }
  }
  wait_vmem();
  barrier();
  store_y(nchunks - 1);

  if (p.final_state) {
    int lo = (nh * NBW * 16 + lg * 4) * P + pc;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MP; ++m)
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = (nh * NBW + jb) * 16 + lg * 4 + r;
          if (m < M && n < N && pc < P)
            p.final_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * P] = S[m][jb][r] * E[m];
        }
  }
}

template <int NB>
constexpr int halves() {
  return NB >= 2 ? 2 : 1;
}

template <typename T>
size_t gtile_bytes(const ScanParams& p) {
  const int64_t nchunks = (p.L + kQ - 1) / kQ;
  return sizeof(T) * (size_t)p.Bsz * nchunks * p.G * kTiles * kTileElems;
}

template <typename T, int NB>
hipError_t launch_cb_variant(const ScanParams& p, T* gt, hipStream_t stream) {
  const int nchunks = (p.L + kQ - 1) / kQ;
  const size_t cb_lds = sizeof(T) * 2 * kQ * (NB * 16 + 8);
  auto cbk = frac_cb_kernel<T, NB>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(cbk), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)cb_lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cbk, dim3(nchunks, p.G, p.Bsz), dim3(256), cb_lds, stream, p, gt);
  return hipGetLastError();
}

template <typename T, int MP, int NB>
hipError_t launch_fwd_variant(const ScanParams& p, void* ws, hipStream_t stream) {
  constexpr int NH = halves<NB>();
  T* gt = reinterpret_cast<T*>(ws);
  hipError_t e = launch_cb_variant<T, NB>(p, gt, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((frac_fwd_kernel<T, MP, NB>), dim3(p.Bsz * p.H), dim3(64 * (p.PP / 16) * NH), 0, stream, p,
                     (const T*)gt);
  return hipGetLastError();
}

template <typename T, int MP>
hipError_t launch_fwd_nb(const ScanParams& p, void* ws, hipStream_t stream) {
  switch (p.NP / 16) {
    case 1: return launch_fwd_variant<T, MP, 1>(p, ws, stream);
    case 2: return launch_fwd_variant<T, MP, 2>(p, ws, stream);
    case 4: return launch_fwd_variant<T, MP, 4>(p, ws, stream);
    case 8: return launch_fwd_variant<T, MP, 8>(p, ws, stream);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch_fwd_mp(const ScanParams& p, void* ws, hipStream_t stream) {
  if (p.M <= 1) return launch_fwd_nb<T, 1>(p, ws, stream);
  if (p.M <= 2) return launch_fwd_nb<T, 2>(p, ws, stream);
  if (p.M <= 4) return launch_fwd_nb<T, 4>(p, ws, stream);
  return launch_fwd_nb<T, 8>(p, ws, stream);
}

}  // namespace

size_t cb_tiles_bytes(const ScanParams& p) {
  if (p.Bsz == 0 || p.L == 0) return 0;
  return p.io_bf16 ? gtile_bytes<bf16>(p) : gtile_bytes<float>(p);
}

hipError_t launch_cb_tiles(const ScanParams& p, void* tiles, hipStream_t stream) {
  const int nb = p.NP / 16;
  if (p.io_bf16) {
    bf16* t = reinterpret_cast<bf16*>(tiles);
    switch (nb) {
      case 1: return launch_cb_variant<bf16, 1>(p, t, stream);
      case 2: return launch_cb_variant<bf16, 2>(p, t, stream);
      case 4: return launch_cb_variant<bf16, 4>(p, t, stream);
      case 8: return launch_cb_variant<bf16, 8>(p, t, stream);
    }
  } else {
    float* t = reinterpret_cast<float*>(tiles);
    switch (nb) {
      case 1: return launch_cb_variant<float, 1>(p, t, stream);
      case 2: return launch_cb_variant<float, 2>(p, t, stream);
      case 4: return launch_cb_variant<float, 4>(p, t, stream);
      case 8: return launch_cb_variant<float, 8>(p, t, stream);
    }
  }
  return hipErrorInvalidValue;
}

size_t scan_fwd_workspace(const ScanParams& p) {
  if (p.Bsz == 0 || p.L == 0) return 0;
  return p.io_bf16 ? gtile_bytes<bf16>(p) : gtile_bytes<float>(p);
}

hipError_t launch_scan_fwd(const ScanParams& p, void* ws, size_t, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  return p.io_bf16 ? launch_fwd_mp<bf16>(p, ws, stream) : launch_fwd_mp<float>(p, ws, stream);
}

}  // namespace frac
