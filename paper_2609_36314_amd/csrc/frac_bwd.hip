// frac_bwd.hip -- chunked parallel scan, backward (training).
//
// Reverse-mode derivative of the selective mode-bank recurrence of Sec. 3.2
// (eq. frac-selective-update, eq. frac-readout, the Appendix-D algorithm), with
// the B/C-widened state, evaluated chunk by chunk like the forward.  Per mode
// (r = 1/tau_m), chunk-local inclusive cumulative step A_t, chunk total A_Q,
// state entering the chunk S0 and adjoint of the chunk's last state G:
//
//   dC_t  = sum_m c_{t,m} e^{-r A_t} S0_m dy_t + sum_{k<=t} Gamma_{t,k} (dy_t . x_k) B_k
//   dx_t  = sum_m kappa_{t,m} e^{-r(A_Q - A_t)} B_t G_m
//           + sum_{t'>=t} Gamma_{t',t} (C_t' . B_t) dy_t' + D dy_t
//   dB_t  = sum_m kappa_{t,m} e^{-r(A_Q - A_t)} G_m x_t
//           + sum_{t'>=t} Gamma_{t',t} (dy_t' . x_t) C_t'
//   G (entering the previous chunk) = e^{-r A_Q} G + sum_t c_{t,m} e^{-r A_t} C_t dy_t^T
//
// and for the step sizes (dc = C^T S dy, dkappa = B^T G x per token and mode):
//   ddtt_t = -sum_m r_m <dS_final, S_final>_m - sum_{t'>=t} e_t' + f_t
//   e_t = sum_m r_m (c dc - kappa dkappa)_{t,m},  f_t = sum_m r_m w rho dkappa_{t,m}
//   ddt_t = ddtt_t * lambda_t^(1/alpha_t)
// (the gradient of the cumulative log-retention telescopes into the suffix sum of
// e).  Inside a chunk the e/f terms reduce to row and column sums of
//   H o Phi and H o Psi,  H = (C B^T) o (dY X^T),
//   Phi_{t,k} = sum_m r_m c_{t,m} kappa_{k,m} e^{-r(A_t - A_k)},
//   Psi_{t,k} = sum_m r_m c_{t,m} w_{k,m} rho_{k,m} e^{-r(A_t - A_k)},
// rank-M products like Gamma.
//
// Three sweeps, each its own kernel; every wave keeps its share of a state or
// adjoint (at most 2 x 4 16x16 float32 tiles per mode group) in matrix-core
// accumulators for the whole sequence:
//   state  forward in time, state transposed (lane = column n of N, rows p): dC
//          (per head), the readout and intra-chunk parts of e and f, the
//          final-state term and sum(dy . x) for dD;
//   rows   reverse, adjoint in row layout (lane = column p of P, rows n): dx and
//          the adjoint parts of e and f;
//   cols   reverse, adjoint transposed (lane = column n): dB (per head).
// The state sweep also writes each chunk's causal tiles (C B^T) o Gamma and
// Gamma o (dY X^T) (bfloat16 for bfloat16 I/O, 10 tiles of 16x16 per chunk and
// head), which the reverse sweeps read instead of forming Gamma again.  With many
// modes and a wide state the state and cols sweeps split N, and the rows sweep
// splits P, over two workgroups per (batch, head), so that no per-head output
// gets a second partial sum.  Tiles are copied straight into
// LDS (natural layout, padded rows) and read back as matrix-core fragments with
// row reads or transposed 64-bit reads.  A finishing kernel forms ddt from the
// suffix sums, and a reduction kernel sums dB and dC over the heads of each group
// in a fixed order.
#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

constexpr int kTiles = 10;
constexpr int kTileElems = 256;
constexpr float kSafeExponent = 55.0f;
constexpr float kRescaleFloor = 0x1p-60f;

__device__ __forceinline__ float uniform(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

// Sum over the 16 lanes of a lane group of v[r] (r = 0..3); returned in every
// lane whose index within the group has ((li >> 2) & 3) == r.  Each step pairs a
// lane with one whose index differs in the step's bit: the mirror lane in the
// 16-lane row (li ^ 15), the mirror in the 8-lane half (li ^ 7), then li ^ 2 and
// li ^ 1, all DPP row permutations; the pairs reached cover the 16 lanes.
__device__ __forceinline__ float reduce16_4(float v[4], int li) {
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const bool hi = li & 8;
    const float send = hi ? v[j] : v[j + 2];
    const float keep = hi ? v[j + 2] : v[j];
    v[j] = keep + dpp_move<0x140>(send);  // row_mirror
  }
  {
    const bool hi = li & 4;
    const float send = hi ? v[0] : v[1];
    const float keep = hi ? v[1] : v[0];
    v[0] = keep + dpp_move<0x141>(send);  // row_half_mirror
  }
  v[0] += dpp_move<0x4E>(v[0]);  // quad_perm [2, 3, 0, 1]
  v[0] += dpp_move<0xB1>(v[0]);  // quad_perm [1, 0, 3, 2]
  return v[0];
}

// ------------------------------------------------------------ shared pieces

template <typename T>
struct Pad {
  static constexpr bool kBf16 = sizeof(T) == 2;
  static constexpr int XS = kBf16 ? 64 + 8 : 64 + 4;  // [t][p] tiles and [t][t'] tiles
  template <int NP>
  static constexpr int BS = kBf16 ? NP + 16 : NP + 8;  // [t][n] tiles read transposed
  template <int NP>
  static constexpr int CS = kBf16 ? NP + 8 : NP + 4;  // [t][n] tiles read along rows
};

// Which sweep computes a chunk's per-(token, mode) weights, and which of them.
enum Role { kState = 0, kRows = 1, kCols = 2 };

// Number of [MP][Q] weight arrays a role keeps in LDS (plus one [Q] array for A_t).
template <int ROLE>
constexpr int n_weight_arrays() {
  return ROLE == kState ? 9 : ROLE == kRows ? 3 : 2;
}

// Per-wave chunk controls (lane = token): effective step, its chunk-local
// inclusive sum and the chunk total.
struct ChunkCtl {
  float dtt, A, al, Alast;
};

__device__ __forceinline__ ChunkCtl chunk_controls(float dtv, float al, float lam, bool has_lambda, int nv) {
  const int lane = threadIdx.x & 63;
  ChunkCtl k;
  const float s_eff = has_lambda ? step_factor(lam, al) : 1.0f;
  k.dtt = (lane < nv) ? dtv * s_eff : 0.0f;
  k.A = wave_inclusive_sum(k.dtt);
  k.Alast = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(k.A), 63));
  k.al = al;
  return k;
}

// Per-(token, mode) weights of one chunk, pair = t * MP + m, written to the
// role's LDS arrays w[i * MP * Q + m * Q + t].  Returns the modes whose chunk
// decay exceeds the factorisation bound (bit m).
//   state: 0 c e^{-rA}, 1 kappa e^{rA} (safe), 2 r c e^{-rA}, 3 r w rho e^{rA} (safe),
//          4 c e^{-rA} E, 5 kappa e^{-r(A_Q-A)} upd, 6 c, 7 kappa, 8 r w rho
//   rows:  0 kappa e^{-r(A_Q-A)} E, 1 r w rho e^{-r(A_Q-A)} E, 2 c e^{-rA} upd
//   cols:  0 kappa e^{-r(A_Q-A)} E, 1 c e^{-rA} upd
// (the reverse sweeps read their Gamma tiles from the state sweep)
// E is the scale of the state (or adjoint) before this chunk's update, upd the
// factor on the update (1/E_new, or 1 when the accumulators are folded back).
template <int MP, int ROLE>
__device__ __forceinline__ int pair_weights(const ChunkCtl& k, int nv, int M, const PairLogits<MP, 512>& lgt,
                                            bool w_is_c, const float* s_rr, const float* s_lnt, const float* Ecur,
                                            float* Enext, float* w) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int j = 0; j < lgt.NPR; ++j) {
    const int pr = tid + 512 * j;
    if (pr >= kQ * MP) break;  // wave-uniform
    const int t = pr / MP, m = pr - t * MP;
    const float A = __shfl(k.A, t, 64), dtt = __shfl(k.dtt, t, 64), al = __shfl(k.al, t, 64);
    const bool valid = t < nv;
    const float r = s_rr[m], prior = -al * s_lnt[m];
    const float zc = (m < M) ? prior + lgt.rl[j] : -INFINITY;
    const float zw = (m < M) ? prior + lgt.wl[j] : -INFINITY;
    // tokens past the sequence get zero weights (their tile rows may hold anything finite)
    const float cw = valid ? group_softmax<MP>(zc) : 0.0f;
    const float ww = w_is_c ? cw : (valid ? group_softmax<MP>(zw) : 0.0f);
    const float xr = r * k.Alast;
    const bool safe = xr <= kSafeExponent;
    const float E = Ecur[m];
    const float Enew = E * fexp(-xr);
    const bool ren = !(Enew >= kRescaleFloor);
    const float upd = ren ? 1.0f : __frcp_rn(Enew);
    const float beta = one_minus_exp_neg(dtt * r);
    const float kap = beta * ww;
    const float ea = fexp(-r * A);
    const float ep = (ROLE == kState && safe) ? fexp(r * A) : 0.0f;
    const float dec = fdecay(r, k.Alast - A);
    float* o = w + m * kWQ + t;
    constexpr int SW = MP * kWQ;  // stride of the weight arrays
    if constexpr (ROLE == kState) {
      const float rwr = r * ww * (1.0f - beta);
      o[0 * SW] = cw * ea;
      o[1 * SW] = kap * ep;
      o[2 * SW] = r * cw * ea;
      o[3 * SW] = rwr * ep;
      o[4 * SW] = cw * ea * E;
      o[5 * SW] = kap * dec * upd;
      o[6 * SW] = cw;
      o[7 * SW] = kap;
      o[8 * SW] = rwr;
    } else if constexpr (ROLE == kRows) {
      o[0 * SW] = kap * dec * E;
      o[1 * SW] = r * ww * (1.0f - beta) * dec * E;
      o[2 * SW] = cw * ea * upd;
    } else {
      o[0 * SW] = kap * dec * E;
      o[1 * SW] = cw * ea * upd;
    }
    if (pr < MP) Enext[m] = ren ? 1.0f : Enew;
  }
  // the same flags in every wave: lane m < MP tests mode m
  const int lane = tid & 63;
  const bool over = lane < MP && lane < M && !(s_rr[lane < MP ? lane : 0] * k.Alast <= kSafeExponent);
  return (int)(__ballot(over) & ((1ull << MP) - 1));
}

// Rank-M product sum_m a[m][row0 + i] b[m][col0 + j] over a 16x16 tile
// (float32 matrix cores, modes as K), in the accumulator layout.
template <int MP>
__device__ __forceinline__ floatx4 rank_m_tile(const float* a, const float* bm, int row0, int col0, int tid = threadIdx.x) {
  const int li = tid & 15, lg = (tid >> 4) & 3;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < (MP + 3) / 4; ++q) {
    const int m = q * 4 + lg;
    const float av = (m < MP) ? a[m * kWQ + row0 + li] : 0.0f;
    const float bv = (m < MP) ? bm[m * kWQ + col0 + li] : 0.0f;
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
  }
  return acc;
}

// Modes past the factorisation bound: add the pairwise-decay terms of
// sum_m a_m[t] b_m[k] s_m e^{-r_m (A_t - A_k)} (t >= k) to a 16x16 tile.
template <int MP>
__device__ __forceinline__ void unsafe_terms(floatx4& acc, int unsafe, const float* a, const float* bm, const float* A,
                                             const float* s_rr, int tb, int kb, bool scale_r, int tid = threadIdx.x) {
  const int li = tid & 15, lg = (tid >> 4) & 3;
  for (int m = 0; m < MP; ++m) {
    if (!((unsafe >> m) & 1)) continue;
    const float rm = s_rr[m];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
      if (t >= k) acc[r] += (scale_r ? rm : 1.0f) * a[m * kWQ + t] * bm[m * kWQ + k] * fdecay(rm, A[t] - A[k]);
    }
  }
}

// dY X^T tile (rows tb, cols kb), K over the 64 columns of P, from natural tiles.
template <typename T, int XS>
__device__ __forceinline__ floatx4 dyx_tile(const T* Ys, const T* Xs, int tb, int kb, int tid = threadIdx.x) {
  const int li = tid & 15, lg = (tid >> 4) & 3;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kp = 0; kp < 2; ++kp) {
    const T* ra = Ys + (tb * 16 + li) * XS + kp * 32 + lg * 4;
    const T* rb = Xs + (kb * 16 + li) * XS + kp * 32 + lg * 4;
    mma(acc, frag_load4x2(ra, ra + 16), frag_load4x2(rb, rb + 16));
  }
  return acc;
}

// Hand-over of partial 16x16 row blocks between the NPART waves that share a
// block of columns: part q finishes the row blocks tb with tb % OW == q (OW =
// min(NPART, 4)); every other part writes its partial of that block to a slot.
template <int NPART>
struct Exchange {
  static constexpr int OW = NPART < 4 ? NPART : 4;
  static constexpr int NSLOT = NPART > 4 ? 4 : 4 - 4 / NPART;
  static constexpr int kFloats = NPART > 1 ? 8 * NSLOT * 256 : 4;
  static __device__ __forceinline__ bool owns(int tb, int part) { return tb % OW == part; }
  static __device__ __forceinline__ int slot(int tb, int part) {
    int s = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j < tb && !owns(j, part)) ++s;
    return s;
  }
  // wave `wave` (part `part`) publishes its non-owned partial blocks
  static __device__ __forceinline__ void put(float* X, int wave, int part, const floatx4* acc) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      if (owns(tb, part)) continue;
      float* dst = X + (wave * NSLOT + slot(tb, part)) * 256;
#pragma unroll
      for (int r = 0; r < 4; ++r) dst[r * 64 + lane] = acc[tb][r];
    }
  }
  // the owner adds the other parts' partials of row block tb, in part order;
  // wave_of(q) is the wave of part q with the same columns
  template <typename F>
  static __device__ __forceinline__ void gather(const float* X, int part, int tb, floatx4& acc, F wave_of) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int q = 0; q < NPART; ++q) {
      if (q == part) continue;
      const float* src = X + (wave_of(q) * NSLOT + slot(tb, q)) * 256;
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] += src[r * 64 + lane];
    }
  }
};

// XCD-aware (batch, head) of a block with PS blocks per head: heads dealt to
// the 8 XCDs in contiguous runs so that heads sharing B and C share an L2.
__device__ __forceinline__ void block_head(int PS, int H, int& b, int& h, int& ps) {
  ps = blockIdx.x % PS;
  int j = blockIdx.x / PS;
  const int nblk = gridDim.x / PS;
  if ((nblk & 7) == 0) j = (j & 7) * (nblk >> 3) + (j >> 3);
  b = j / H;
  h = j - b * H;
}

struct BwdWork {
  const void* tiles;  // C B^T tiles
  void* gg;           // (C B^T) o Gamma per (batch, chunk, head), causal tiles in fragment order
  void* hg;           // Gamma o (dY X^T), the same layout
  void* dBp;          // per-head dB, [B, L, H, N]
  void* dCp;          // per-head dC
  float* eA;          // [2][B H L] readout / intra part of e (per N half)
  float* fA;          // [2][B H L] intra part of f (per N half)
  float* eB;          // [2][B H L] adjoint part of e (per P half)
  float* fB;          // [2][B H L] adjoint part of f
  float* F;           // [2][B H] final-state term (per N half)
  float* dDp;         // [B H] sum(dy . x)
  float* tsum;        // [B H][L / 64] totals of e over 64-token tiles
};

// ------------------------------------------------ state / cols sweep layout

// Transposed layout (lane = column n): the workgroup holds NBF 16-column blocks
// of N (all of N, or half when MP * NB > 32); its 8 waves are those blocks times
// FPART parts, the parts splitting the modes.
template <typename T, int MP, int NB>
struct ColCfg {
  static constexpr int NP = NB * 16;
  static constexpr int XS = Pad<T>::XS;
  static constexpr int BS = Pad<T>::template BS<NP>;
  static constexpr int CS = Pad<T>::template CS<NP>;
  static constexpr int PS = MP * NB > 32 ? 2 : 1;
  static constexpr int NBF = NB / PS;
  static constexpr int FPART = 8 / NBF;
  static constexpr int MPF = MP >= FPART ? MP / FPART : 1;
  static constexpr int NACT = MP >= FPART ? FPART : MP;  // parts holding modes (the rest idle)
  static constexpr int NBUF = Pad<T>::kBf16 ? 2 : 1;
};

// ------------------------------------------------------------ state sweep

template <typename T, int MP, int NB>
__global__ void __launch_bounds__(512) frac_bwd_state_kernel(ScanParams p, BwdWork wk) {
  using Cfg = ColCfg<T, MP, NB>;
  constexpr int NP = Cfg::NP, XS = Cfg::XS, BS = Cfg::BS, CS = Cfg::CS;
  constexpr int NBF = Cfg::NBF, FPART = Cfg::FPART, MPF = Cfg::MPF;
  using Ex = Exchange<Cfg::NACT>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M, G = p.G;
  const int nchunks = (L + kQ - 1) / kQ;
  int b, h, ps;
  block_head(Cfg::PS, H, b, h, ps);
  const int g = h * G / H;
  const int nbl = wave % NBF, part = wave / NBF, nb = ps * NBF + nbl, ncol = nb * 16 + li;
  const int mo = part * MPF;
  const bool active = mo < MP;

  __shared__ __align__(16) T Xb0[64 * XS], Yb0[64 * XS], Bb0[64 * BS];
  __shared__ __align__(16) T Xb1[Cfg::NBUF == 2 ? 64 * XS : 8], Yb1[Cfg::NBUF == 2 ? 64 * XS : 8],
      Bb1[Cfg::NBUF == 2 ? 64 * BS : 8];
  __shared__ __align__(16) T Cb[64 * CS];
  constexpr int NWA = n_weight_arrays<kState>();
  constexpr int oHG = 0;                                         // T [k][t] (Gamma o dY X^T)^T, causal
  constexpr int WSZ = NWA * MP * kWQ + kQ;                        // one chunk's weights [NWA][MP][Q], A [Q]
  // two chunks' weights (the next one formed during this one's update) when LDS allows
  constexpr int kTileBytes = (Cfg::NBUF * 64 * (2 * XS + BS) + 64 * CS) * (int)sizeof(T);
  constexpr int kFixed = 64 * XS * (int)sizeof(T) + (3 * kTiles * 16 + 8 * kQ + Ex::kFloats + 4 * MP) * 4;
  constexpr int NWB = kTileBytes + kFixed + 2 * WSZ * 4 <= 160 * 1024 - 512 ? 2 : 1;
  constexpr int oW = oHG + 64 * XS * (int)sizeof(T);             // float weights, NWB chunks
  constexpr int oSl = oW + NWB * WSZ * 4;                        // float slots R, C, F [10][16] each
  constexpr int oRd = oSl + 3 * kTiles * 16 * 4;                 // float [8][Q] per-wave token partials
  constexpr int oEx = oRd + 8 * kQ * 4;                          // float exchange
  constexpr int oSc = oEx + Ex::kFloats * 4;                     // float rates, log tau, scales
  __shared__ __align__(16) unsigned char sm[oSc + 4 * MP * 4];
  T* HGT = reinterpret_cast<T*>(sm + oHG);
  float* const W0 = reinterpret_cast<float*>(sm + oW);
  float* const W1 = W0 + (NWB - 1) * WSZ;
  float* slotR = reinterpret_cast<float*>(sm + oSl);
  float* slotC = slotR + kTiles * 16;
  float* slotF = slotC + kTiles * 16;
  float* redR = reinterpret_cast<float*>(sm + oRd);
  float* XCH = reinterpret_cast<float*>(sm + oEx);
  float* s_rr = reinterpret_cast<float*>(sm + oSc);
  float* s_lnt = s_rr + MP;
  float* s_E2 = s_lnt + MP;
  constexpr int SW = MP * kWQ;  // stride of the weight arrays

  if (tid < MP) {
    const float tau = (tid < M) ? p.tau[tid] : 1.0f;
    s_rr[tid] = (tid < M) ? 1.0f / tau : 0.0f;
    s_lnt[tid] = (tid < M) ? logf(tau) : 0.0f;
    s_E2[tid] = 1.0f;
  }
  for (int i = tid; i < 64 * XS; i += 512) {
    HGT[i] = (T)0.0f;
    Xb0[i] = Yb0[i] = (T)0.0f;
    Xb1[Cfg::NBUF == 2 ? i : 0] = Yb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;
  }
  for (int i = tid; i < 64 * BS; i += 512) Bb0[i] = Bb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;
  for (int i = tid; i < 64 * CS; i += 512) Cb[i] = (T)0.0f;

  // ---- state S^T: S[m][pb] holds mode mo + m, rows p = 16 pb + 4 lg + r, column ncol
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)M * N * P;
  floatx4 S[MPF][4];
  {
    int lo = ncol * P + lg * 4;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MPF; ++m)
#pragma unroll
      for (int pb = 0; pb < 4; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pr = pb * 16 + lg * 4 + r;
          float v = 0.0f;
          if (p.init_state && active && mo + m < M && ncol < N && pr < P)
            v = p.init_state[sbase + (int64_t)(mo + m) * N * P + lo + pb * 16 + r];
          S[m][pb][r] = v;
        }
  }

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * P;
  const T* yg = reinterpret_cast<const T*>(p.dy) + (((int64_t)b * L) * H + h) * P;
  const T* Bgp = reinterpret_cast<const T*>(p.Bm) + (((int64_t)b * L) * G + g) * N;
  const T* Cgp = reinterpret_cast<const T*>(p.Cm) + (((int64_t)b * L) * G + g) * N;
  const int64_t xstride = (int64_t)H * P, bstride = (int64_t)G * N;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const int64_t lg_st = (int64_t)H * M;
  PairLogits<MP, 512> lgt_n;  // the logits of the next chunk's weight pass
  auto load_controls = [&](int c, float& dtv, float& al, float& lam) {
    const int tg = c * kQ + lane;
    const bool valid = tg < L;
    dtv = valid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al = valid ? al_bh[tg * p.as1] : 1.0f;
    lam = (valid && lm_bh) ? lm_bh[tg * p.ls1] : 1.0f;
    lgt_n.load(rl_bh, wl_bh, c * kQ, min(kQ, L - c * kQ), M, lg_st, threadIdx.x);
  };
  DmaPlan<T, XS> planX;
  DmaPlan<T, BS> planB;
  DmaPlan<T, CS> planC;
  planX.init(xstride, P);
  planB.init(bstride, N);
  planC.init(bstride, N);
  auto stage = [&](int c, T* Xd, T* Yd, T* Bd) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    planX.issue_async(Xd, xg + (int64_t)t0 * xstride, xstride, nv);
    planX.issue_async(Yd, yg + (int64_t)t0 * xstride, xstride, nv);
    planB.issue_async(Bd, Bgp + (int64_t)t0 * bstride, bstride, nv);
  };
  auto stageC = [&](int c) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    planC.issue_async(Cb, Cgp + (int64_t)t0 * bstride, bstride, nv);
  };

  float dt_n, al_n, lam_n;
  load_controls(0, dt_n, al_n, lam_n);
  if (Cfg::NBUF == 2) {
    stage(0, Xb0, Yb0, Bb0);
    stageC(0);
  }
  float dd_acc = 0.0f;
  const T* gtiles = reinterpret_cast<const T*>(wk.tiles);
  TilePrefetch<T> gtile;  // C B^T tile values, loaded one chunk ahead
  gtile.load(gtiles + ((int64_t)b * nchunks * G + g) * (kTiles * kTileElems), wave, lane);
  T* dCp = reinterpret_cast<T*>(wk.dCp);
  const int64_t bl_h = (int64_t)p.Bsz * L * H;

  // Per-(token, mode) weights of chunk c into Wd, from the controls in dt_n, al_n,
  // lam_n.  Chunk c + 1's weights are formed at the end of chunk c's step, so that
  // their latency overlaps that step's state update.
  float alast_c = 0.0f;  // chunk total of the effective steps
  int unsafe_c = 0;      // modes past the factorisation bound
  auto weights = [&](int c, float* Wd) __attribute__((always_inline)) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    const ChunkCtl k = chunk_controls(dt_n, al_n, lam_n, lm_bh != nullptr, nv);
    if (wave == 0) Wd[NWA * MP * kWQ + lane] = k.A;
    unsafe_c = pair_weights<MP, kState>(k, nv, M, lgt_n, rl_bh == wl_bh, s_rr, s_lnt, s_E2 + (c & 1) * MP,
                                        s_E2 + ((c + 1) & 1) * MP, Wd);
    alast_c = k.Alast;
  };
  barrier();  // rates and scales in LDS
  if constexpr (NWB == 2) weights(0, W0);

  auto step = [&](int c, T* Xc, T* Yc, T* Bc, T* Xn, T* Yn, T* Bn, float* W, float* Wn)
                  __attribute__((always_inline)) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    // lane-derived addresses recomputed per chunk rather than held across the loop
    const int tid = fresh_tid(), lane = tid & 63, li = lane & 15, lg = lane >> 4;
    const float* Ecur = s_E2 + (c & 1) * MP;
    const float* P_O = W;
    const float* P_Vt = W + 1 * SW;
    const float* P_rO = W + 2 * SW;
    const float* P_Y = W + 3 * SW;
    const float* P_wdc = W + 4 * SW;  // times r_m: the readout weight of e
    const float* P_v = W + 5 * SW;
    const float* P_c = W + 6 * SW;
    const float* P_k = W + 7 * SW;
    const float* P_wr = W + 8 * SW;
    const float* P_A = W + NWA * MP * kWQ;
    wait_vmem();
    barrier();  // this chunk's tiles and weights have landed; the previous chunk is done
    const TilePrefetch<T> gcur = gtile.pinned_copy();  // before any new memory operation
    if (Cfg::NBUF == 2) {
      if (c + 1 < nchunks) stage(c + 1, Xn, Yn, Bn);
    } else {
      stage(c, Xc, Yc, Bc);
      stageC(c);
      wait_vmem();
      barrier();
    }
    if constexpr (NWB == 1) weights(c, W);
    if (c + 1 < nchunks) load_controls(c + 1, dt_n, al_n, lam_n);
    if constexpr (NWB == 1) barrier();  // weights in LDS
    const int unsafe = unsafe_c;
    float renf[MPF];
    int renbits = 0;
#pragma unroll
    for (int m = 0; m < MPF; ++m) {
      const float Enew = uniform(Ecur[mo + m] * fexp(-s_rr[mo + m] * alast_c));
      renf[m] = Enew;
      if (__float_as_int(Enew) < __float_as_int(kRescaleFloor)) renbits |= 1 << m;
    }

    __builtin_amdgcn_sched_barrier(0);
    // ---- intra-chunk tiles: HG = Gamma o D (LDS, transposed), row / column sums of
    // H o Phi and column sums of H o Psi (first workgroup of the head only)
    {
#pragma unroll
      for (int jt = 0; jt < 2; ++jt) {
        const int tile = wave + 8 * jt;
        if (tile >= kTiles) break;
        const int tb = tile_row(tile), kb = tile_col(tile);
        const floatx4 D = dyx_tile<T, XS>(Yc, Xc, tb, kb, tid);
        floatx4 Gm = rank_m_tile<MP>(P_O, P_Vt, tb * 16, kb * 16, tid);
        if (unsafe) unsafe_terms<MP>(Gm, unsafe, P_c, P_k, P_A, s_rr, tb, kb, false, tid);
        float hv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r, kk = kb * 16 + li;
          hv[r] = keep_if_ge(Gm[r] * D[r], t, kk);
        }
        T* dst = HGT + (kb * 16 + li) * XS + tb * 16 + lg * 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[r] = (T)hv[r];
        {  // the tiles of the reverse sweeps, once per head: (C B^T) o Gamma from the
           // first workgroup of the head, Gamma o (dY X^T) from the last
          const int64_t to = ((int64_t)(b * nchunks + c) * H + h) * (kTiles * kTileElems) + tile * kTileElems + lane * 4;
          if (ps == 0) {
            floatx4 gv;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int t = tb * 16 + lg * 4 + r, kk = kb * 16 + li;
              gv[r] = keep_if_ge(gcur.get(jt, r) * Gm[r], t, kk);
            }
            store4(reinterpret_cast<T*>(wk.gg) + to, gv);
          }
          if (ps == Cfg::PS - 1) store4(reinterpret_cast<T*>(wk.hg) + to, floatx4{hv[0], hv[1], hv[2], hv[3]});
        }
        if (tile % Cfg::PS == ps) {  // the two halves of N share the tile sums
          floatx4 Ph = rank_m_tile<MP>(P_rO, P_Vt, tb * 16, kb * 16, tid);
          floatx4 Ps = rank_m_tile<MP>(P_O, P_Y, tb * 16, kb * 16, tid);
          if (unsafe) {
            unsafe_terms<MP>(Ph, unsafe, P_c, P_k, P_A, s_rr, tb, kb, true, tid);
            unsafe_terms<MP>(Ps, unsafe, P_c, P_wr, P_A, s_rr, tb, kb, false, tid);
          }
          float rv[4], ce = 0.f, cf = 0.f;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = tb * 16 + lg * 4 + r, kk = kb * 16 + li;
            const float hm = keep_if_ge(gcur.get(jt, r) * D[r], t, kk);
            rv[r] = hm * Ph[r];
            ce += hm * Ph[r];
            cf += hm * Ps[r];
          }
          const float rs = reduce16_4(rv, li);
          if ((li & 3) == 0) slotR[tile * 16 + lg * 4 + ((li >> 2) & 3)] = rs;
          ce = xor32_sum(xor16_sum(ce));
          cf = xor32_sum(xor16_sum(cf));
          if (lg == 0) {
            slotC[tile * 16 + li] = ce;
            slotF[tile * 16 + li] = cf;
          }
        }
      }
    }

    if (c + 1 < nchunks) gtile.load(gtiles + (((int64_t)b * nchunks + c + 1) * G + g) * (kTiles * kTileElems), wave, lane);

    __builtin_amdgcn_sched_barrier(0);
    // ---- readout side of the state entering the chunk, transposed: U^T_m = S_m dY^T
    // (rows n of this wave's block, columns t), dC^T (inter) and the readout part of e
    floatx4 dCa[4];  // dC^T: rows n = 16 nb + 4 lg + r, column t = 16 tb + li
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) dCa[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    {
      float racc[4] = {0.f, 0.f, 0.f, 0.f};  // per row block: this lane's token
      if (active) {
        Frag<T> Sa[MPF][2];
#pragma unroll
        for (int m = 0; m < MPF; ++m)
#pragma unroll
          for (int kp = 0; kp < 2; ++kp) {
#pragma unroll
            for (int s = 0; s < 4; ++s) frag_set(Sa[m][kp], s, S[m][2 * kp][s]);
#pragma unroll
            for (int s = 0; s < 4; ++s) frag_set(Sa[m][kp], 4 + s, S[m][2 * kp + 1][s]);
          }
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
          const T* row = Yc + (tb * 16 + li) * XS + lg * 4;
          const Frag<T> y0 = frag_load4x2(row, row + 16), y1 = frag_load4x2(row + 32, row + 48);
          floatx4 ws = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int m = 0; m < MPF; ++m) {
            floatx4 U = {0.f, 0.f, 0.f, 0.f};
            mma(U, Sa[m][0], y0);
            mma(U, Sa[m][1], y1);
            const float wd = P_wdc[(mo + m) * kWQ + tb * 16 + li];
            const float rm = s_rr[mo + m];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float v = wd * U[r];
              dCa[tb][r] += v;
              ws[r] += rm * v;
            }
          }
          // sum over n of C_t[n] ws[n]: this lane's 4 values, then the 4 lane groups
          const T* crow = Cb + (tb * 16 + li) * CS + nb * 16 + lg * 4;
          float cv[4];
          load4(crow, cv);
          racc[tb] = ws[0] * cv[0] + ws[1] * cv[1] + ws[2] * cv[2] + ws[3] * cv[3];
        }
        if (Cfg::NACT > 1) Ex::put(XCH, wave, part, dCa);
      }
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        float v = racc[tb];
        v = xor32_sum(xor16_sum(v));
        if (lg == 0) redR[wave * kQ + tb * 16 + li] = v;
      }
    }
    barrier();  // HG, slots, token partials and exchange complete; C is free
    if (Cfg::NBUF == 2 && c + 1 < nchunks) stageC(c + 1);

    if (wave == 0) {
      // token t: readout part (all waves) [+ row sums of its row-block tiles - column
      // sums of its column-block tiles], fixed order
      const int t = lane, tbt = t >> 4, tr = t & 15;
      float er = 0.f, ec = 0.f, ef = 0.f;
      for (int w2 = 0; w2 < 8; ++w2) er += redR[w2 * kQ + t];
      for (int kb2 = 0; kb2 <= tbt; ++kb2) {
        const int tile = tbt * (tbt + 1) / 2 + kb2;
        if (tile % Cfg::PS == ps) er += slotR[tile * 16 + tr];
      }
      for (int tb2 = tbt; tb2 < 4; ++tb2) {
        const int tile = tb2 * (tb2 + 1) / 2 + tbt;
        if (tile % Cfg::PS == ps) {
          ec += slotC[tile * 16 + tr];
          ef += slotF[tile * 16 + tr];
        }
      }
      if (t < nv) {
        const int64_t ith = ((int64_t)b * H + h) * L + t0 + t;  // [B, H, L]: one head's tokens contiguous
        wk.eA[ps * bl_h + ith] = er - ec;
        wk.fA[ps * bl_h + ith] = ef;
      }
    }
    if (ps == 0 && p.dD) {
      // sum(dy . x) of the chunk for dD: 8 consecutive columns of one token per
      // thread (columns past P hold zeros)
      const int t = tid >> 3, c8 = (tid & 7) * 8;
      if (t < nv) {
        float xv[8], yv[8];
        load8(Xc + t * XS + c8, xv);
        load8(Yc + t * XS + c8, yv);
#pragma unroll
        for (int j = 0; j < 8; ++j) dd_acc += xv[j] * yv[j];
      }
    }
    if (active) {  // waves holding state

    __builtin_amdgcn_sched_barrier(0);
    // ---- dC^T blocks this wave finishes: other parts + intra B^T (Gamma o dY X^T)^T, causal
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      if (!Ex::owns(tb, part)) continue;
      if (Cfg::NACT > 1) Ex::gather(XCH, part, tb, dCa[tb], [&](int q) { return q * NBF + nbl; });
#pragma unroll
      for (int kk = 0; kk <= tb / 2; ++kk) {
        const Frag<T> a = frag_load_rows(Bc, BS, kk * 32 + lg * 8, nb * 16, tid);
        const Frag<T> bb = frag_load_rows(HGT, XS, kk * 32 + lg * 8, tb * 16, tid);
        mma(dCa[tb], a, bb);
      }
      // per-head partial: token t = 16 tb + li, columns n .. n+3 (32-bit offsets from the chunk)
      const int t = tb * 16 + li, n = nb * 16 + lg * 4;
      if (t < nv && n < N) store4(dCp + (((int64_t)b * L + t0) * H + h) * N + t * (H * N) + n, dCa[tb]);
    }

    __builtin_amdgcn_sched_barrier(0);
    // ---- state update S^T += X^T (v o B), rows p, column ncol
#pragma unroll
    for (int m = 0; m < MPF; ++m) {
      if (!((renbits >> m) & 1)) continue;
#pragma unroll
      for (int pb = 0; pb < 4; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) S[m][pb][r] *= renf[m];
    }
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      Frag<T> Xa[4];
#pragma unroll
      for (int pb = 0; pb < 4; ++pb) Xa[pb] = frag_load_rows(Xc, XS, kt * 32 + lg * 8, pb * 16, tid);
      const Frag<T> bf = frag_load_rows(Bc, BS, kt * 32 + lg * 8, nb * 16, tid);
      float b8[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) b8[s] = to_f32(bf.v[s]);
#pragma unroll
      for (int m = 0; m < MPF; ++m) {
        const float* pv = P_v + (mo + m) * kWQ + kt * 32 + lg * 8;
        const float4 v0 = *reinterpret_cast<const float4*>(pv);
        const float4 v1 = *reinterpret_cast<const float4*>(pv + 4);
        Frag<T> Bv;
        frag_set(Bv, 0, b8[0] * v0.x);
        frag_set(Bv, 1, b8[1] * v0.y);
        frag_set(Bv, 2, b8[2] * v0.z);
        frag_set(Bv, 3, b8[3] * v0.w);
        frag_set(Bv, 4, b8[4] * v1.x);
        frag_set(Bv, 5, b8[5] * v1.y);
        frag_set(Bv, 6, b8[6] * v1.z);
        frag_set(Bv, 7, b8[7] * v1.w);
#pragma unroll
        for (int pb = 0; pb < 4; ++pb) mma(S[m][pb], Xa[pb], Bv);
      }
    }
    }  // active
    if constexpr (NWB == 2) {
      if (c + 1 < nchunks) weights(c + 1, Wn);
    }
  };

  for (int c = 0; c < nchunks; c += 2) {
    step(c, Xb0, Yb0, Bb0, Xb1, Yb1, Bb1, W0, W1);
    if (c + 1 < nchunks) {
      if (Cfg::NBUF == 2) step(c + 1, Xb1, Yb1, Bb1, Xb0, Yb0, Bb0, W1, W0);
      else step(c + 1, Xb0, Yb0, Bb0, Xb0, Yb0, Bb0, W1, W0);
    }
  }
  wait_vmem();
  barrier();

  // ---- final-state term sum_m r_m <dS_final_m, S_final_m> and sum(dy . x)
  float fpart = 0.0f;
  if (p.d_final_state && active) {
    const float* Ef = s_E2 + (nchunks & 1) * MP;
    int lo = ncol * P + lg * 4;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MPF; ++m) {
      const float scale = (mo + m < M) ? s_rr[mo + m] * Ef[mo + m] : 0.0f;
#pragma unroll
      for (int pb = 0; pb < 4; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pr = pb * 16 + lg * 4 + r;
          if (mo + m < M && ncol < N && pr < P)
            fpart += scale * S[m][pb][r] * p.d_final_state[sbase + (int64_t)(mo + m) * N * P + lo + pb * 16 + r];
        }
    }
  }
  float* red = reinterpret_cast<float*>(sm + oW);  // the weights are no longer needed
  red[tid] = fpart;
  red[512 + tid] = dd_acc;
  barrier();
  if (tid == 0) {
    float fs = 0.f, ds = 0.f;
    for (int i = 0; i < 512; ++i) {
      fs += red[i];
      ds += red[512 + i];
    }
    wk.F[(int64_t)ps * p.Bsz * H + (int64_t)b * H + h] = fs;
    if (ps == 0) wk.dDp[(int64_t)b * H + h] = ds;
  }
}

// ------------------------------------------------------------- cols sweep

template <typename T, int MP, int NB>
__global__ void __launch_bounds__(512) frac_bwd_cols_kernel(ScanParams p, BwdWork wk) {
  using Cfg = ColCfg<T, MP, NB>;
  constexpr int NP = Cfg::NP, XS = Cfg::XS, CS = Cfg::BS;  // C is read transposed here
  constexpr int NBF = Cfg::NBF, FPART = Cfg::FPART, MPF = Cfg::MPF;
  using Ex = Exchange<Cfg::NACT>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M, G = p.G;
  const int nchunks = (L + kQ - 1) / kQ;
  int b, h, ps;
  block_head(Cfg::PS, H, b, h, ps);
  const int g = h * G / H;
  const int nbl = wave % NBF, part = wave / NBF, nb = ps * NBF + nbl, ncol = nb * 16 + li;
  const int mo = part * MPF;
  const bool active = mo < MP;

  __shared__ __align__(16) T Xb0[64 * XS], Yb0[64 * XS], Cb0[64 * CS];
  __shared__ __align__(16) T Xb1[Cfg::NBUF == 2 ? 64 * XS : 8], Yb1[Cfg::NBUF == 2 ? 64 * XS : 8],
      Cb1[Cfg::NBUF == 2 ? 64 * CS : 8];
  constexpr int NWA = n_weight_arrays<kCols>();
  constexpr int oHG = 0;                                         // T [t][k] Gamma o dY X^T, causal
  constexpr int oW = oHG + 64 * XS * (int)sizeof(T);
  constexpr int oEx = oW + (NWA * MP * kWQ + kQ) * 4;
  constexpr int oSc = oEx + Ex::kFloats * 4;
  __shared__ __align__(16) unsigned char sm[oSc + 4 * MP * 4];
  T* HG = reinterpret_cast<T*>(sm + oHG);
  float* W = reinterpret_cast<float*>(sm + oW);
  float* P_A = W + NWA * MP * kWQ;
  float* XCH = reinterpret_cast<float*>(sm + oEx);
  float* s_rr = reinterpret_cast<float*>(sm + oSc);
  float* s_lnt = s_rr + MP;
  float* s_E2 = s_lnt + MP;
  constexpr int SW = MP * kWQ;  // stride of the weight arrays
  const float* P_wdb = W;
  const float* P_om = W + 1 * SW;

  if (tid < MP) {
    const float tau = (tid < M) ? p.tau[tid] : 1.0f;
    s_rr[tid] = (tid < M) ? 1.0f / tau : 0.0f;
    s_lnt[tid] = (tid < M) ? logf(tau) : 0.0f;
    s_E2[tid] = 1.0f;
  }
  for (int i = tid; i < 64 * XS; i += 512) {
    HG[i] = (T)0.0f;
    Xb0[i] = Yb0[i] = (T)0.0f;
    Xb1[Cfg::NBUF == 2 ? i : 0] = Yb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;
  }
  for (int i = tid; i < 64 * CS; i += 512) Cb0[i] = Cb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;

  // ---- adjoint G^T: Gs[m][pb] holds mode mo + m, rows p = 16 pb + 4 lg + r, column ncol
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)M * N * P;
  floatx4 Gs[MPF][4];
  {
    int lo = ncol * P + lg * 4;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MPF; ++m)
#pragma unroll
      for (int pb = 0; pb < 4; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pr = pb * 16 + lg * 4 + r;
          float v = 0.0f;
          if (p.d_final_state && active && mo + m < M && ncol < N && pr < P)
            v = p.d_final_state[sbase + (int64_t)(mo + m) * N * P + lo + pb * 16 + r];
          Gs[m][pb][r] = v;
        }
  }

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * P;
  const T* yg = reinterpret_cast<const T*>(p.dy) + (((int64_t)b * L) * H + h) * P;
  const T* Cgp = reinterpret_cast<const T*>(p.Cm) + (((int64_t)b * L) * G + g) * N;
  const int64_t xstride = (int64_t)H * P, bstride = (int64_t)G * N;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const int64_t lg_st = (int64_t)H * M;
  PairLogits<MP, 512> lgt_n;  // the logits of the next chunk's weight pass
  auto load_controls = [&](int c, float& dtv, float& al, float& lam) {
    const int tg = c * kQ + lane;
    const bool valid = tg < L;
    dtv = valid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al = valid ? al_bh[tg * p.as1] : 1.0f;
    lam = (valid && lm_bh) ? lm_bh[tg * p.ls1] : 1.0f;
    lgt_n.load(rl_bh, wl_bh, c * kQ, min(kQ, L - c * kQ), M, lg_st, threadIdx.x);
  };
  DmaPlan<T, XS> planX;
  DmaPlan<T, CS> planC;
  planX.init(xstride, P);
  planC.init(bstride, N);
  // (LDS addresses passed opaquely: the compiler otherwise folds the address-space
  // conversion of these tiles into an instruction it cannot encode)
  auto stage = [&](int c, T* Xd, T* Yd, T* Cd) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    planX.issue_async(Xd, xg + (int64_t)t0 * xstride, xstride, nv);
    planX.issue_async(Yd, yg + (int64_t)t0 * xstride, xstride, nv);
    planC.issue_async(Cd, Cgp + (int64_t)t0 * bstride, bstride, nv);
  };

  float dt_n, al_n, lam_n;
  load_controls(nchunks - 1, dt_n, al_n, lam_n);
  if (Cfg::NBUF == 2) stage(nchunks - 1, Xb0, Yb0, Cb0);
  T* dBp = reinterpret_cast<T*>(wk.dBp);
  // Gamma o (dY X^T) tiles written by the state sweep, loaded one chunk ahead (in processing order)
  const T* hgtiles = reinterpret_cast<const T*>(wk.hg);
  TilePrefetch<T> hgt;
  hgt.load(hgtiles + ((int64_t)(b * nchunks + nchunks - 1) * H + h) * (kTiles * kTileElems), wave, lane);

  // chunks in reverse order; i counts processed chunks (buffer parity)
  auto step = [&](int c, int i, T* Xc, T* Yc, T* Cc, T* Xn, T* Yn, T* Cn) __attribute__((always_inline)) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    const float* Ecur = s_E2 + (i & 1) * MP;
    float* Enext = s_E2 + ((i + 1) & 1) * MP;
    wait_vmem();
    barrier();
    // this chunk's prefetched controls, logits and tile values, taken before any new memory operation
    const float dtv = pinned(dt_n), al_l = pinned(al_n), lam_l = pinned(lam_n);
    const PairLogits<MP, 512> lgt = lgt_n.pinned_copy();
    const TilePrefetch<T> hcur = hgt.pinned_copy();
    if (Cfg::NBUF == 2) {
      if (c > 0) stage(c - 1, Xn, Yn, Cn);
    } else {
      stage(c, Xc, Yc, Cc);
      wait_vmem();
      barrier();
    }
    if (c > 0) load_controls(c - 1, dt_n, al_n, lam_n);
    const ChunkCtl k = chunk_controls(dtv, al_l, lam_l, lm_bh != nullptr, nv);
    if (wave == 0) P_A[lane] = k.A;
    const int unsafe = pair_weights<MP, kCols>(k, nv, M, lgt, rl_bh == wl_bh, s_rr, s_lnt, Ecur, Enext, W);
    float renf[MPF];
    int renbits = 0;
#pragma unroll
    for (int m = 0; m < MPF; ++m) {
      const float Enew = uniform(Ecur[mo + m] * fexp(-s_rr[mo + m] * k.Alast));
      renf[m] = Enew;
      if (__float_as_int(Enew) < __float_as_int(kRescaleFloor)) renbits |= 1 << m;
    }
    barrier();  // weights in LDS

    __builtin_amdgcn_sched_barrier(0);
    // ---- HG = Gamma o dY X^T (natural [t][k], causal)
#pragma unroll
    for (int jt = 0; jt < 2; ++jt) {
      const int tile = wave + 8 * jt;
      if (tile >= kTiles) break;
      const int tb = tile_row(tile), kb = tile_col(tile);
#pragma unroll
      for (int r = 0; r < 4; ++r) HG[(tb * 16 + lg * 4 + r) * XS + kb * 16 + li] = hcur.v[jt].e[r];
    }
    (void)unsafe;
    if (c > 0) hgt.load(hgtiles + ((int64_t)(b * nchunks + c - 1) * H + h) * (kTiles * kTileElems), wave, lane);

    __builtin_amdgcn_sched_barrier(0);
    // ---- V^T_m = G_m X^T (rows n of this wave's block, columns k) -> dB^T (inter)
    floatx4 dBa[4];  // dB^T: rows n = 16 nb + 4 lg + r, column k = 16 tb + li
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) dBa[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (active) {
      Frag<T> Ga[MPF][2];
#pragma unroll
      for (int m = 0; m < MPF; ++m)
#pragma unroll
        for (int kp = 0; kp < 2; ++kp) {
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Ga[m][kp], s, Gs[m][2 * kp][s]);
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Ga[m][kp], 4 + s, Gs[m][2 * kp + 1][s]);
        }
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        const T* row = Xc + (tb * 16 + li) * XS + lg * 4;
        const Frag<T> x0 = frag_load4x2(row, row + 16), x1 = frag_load4x2(row + 32, row + 48);
#pragma unroll
        for (int m = 0; m < MPF; ++m) {
          floatx4 V = {0.f, 0.f, 0.f, 0.f};
          mma(V, Ga[m][0], x0);
          mma(V, Ga[m][1], x1);
          const float wb = P_wdb[(mo + m) * kWQ + tb * 16 + li];
#pragma unroll
          for (int r = 0; r < 4; ++r) dBa[tb][r] += wb * V[r];
        }
      }
      if (Cfg::NACT > 1) Ex::put(XCH, wave, part, dBa);
    }
    barrier();  // HG and exchange complete
    if (!active) return;

    __builtin_amdgcn_sched_barrier(0);
    // ---- dB^T blocks this wave finishes: other parts + intra C^T (Gamma o dY X^T), t >= k
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      if (!Ex::owns(tb, part)) continue;
      if (Cfg::NACT > 1) Ex::gather(XCH, part, tb, dBa[tb], [&](int q) { return q * NBF + nbl; });
#pragma unroll
      for (int kk = tb / 2; kk < 2; ++kk) {
        const Frag<T> a = frag_load_rows(Cc, CS, kk * 32 + lg * 8, nb * 16);
        const Frag<T> bb = frag_load_rows(HG, XS, kk * 32 + lg * 8, tb * 16);
        mma(dBa[tb], a, bb);
      }
      const int k = tb * 16 + li, n = nb * 16 + lg * 4;
      if (k < nv && n < N) store4(dBp + (((int64_t)b * L + t0) * H + h) * N + k * (H * N) + n, dBa[tb]);
    }

    __builtin_amdgcn_sched_barrier(0);
    // ---- adjoint update G^T += dY^T (omega o C), rows p, column ncol
#pragma unroll
    for (int m = 0; m < MPF; ++m) {
      if (!((renbits >> m) & 1)) continue;
#pragma unroll
      for (int pb = 0; pb < 4; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) Gs[m][pb][r] *= renf[m];
    }
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      Frag<T> Ya[4];
#pragma unroll
      for (int pb = 0; pb < 4; ++pb) Ya[pb] = frag_load_rows(Yc, XS, kt * 32 + lg * 8, pb * 16);
      const Frag<T> cf = frag_load_rows(Cc, CS, kt * 32 + lg * 8, nb * 16);
      float c8[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) c8[s] = to_f32(cf.v[s]);
#pragma unroll
      for (int m = 0; m < MPF; ++m) {
        const float* pv = P_om + (mo + m) * kWQ + kt * 32 + lg * 8;
        const float4 v0 = *reinterpret_cast<const float4*>(pv);
        const float4 v1 = *reinterpret_cast<const float4*>(pv + 4);
        Frag<T> Cv;
        frag_set(Cv, 0, c8[0] * v0.x);
        frag_set(Cv, 1, c8[1] * v0.y);
        frag_set(Cv, 2, c8[2] * v0.z);
        frag_set(Cv, 3, c8[3] * v0.w);
        frag_set(Cv, 4, c8[4] * v1.x);
        frag_set(Cv, 5, c8[5] * v1.y);
        frag_set(Cv, 6, c8[6] * v1.z);
        frag_set(Cv, 7, c8[7] * v1.w);
#pragma unroll
        for (int pb = 0; pb < 4; ++pb) mma(Gs[m][pb], Ya[pb], Cv);
      }
    }
  };

  for (int i = 0; i < nchunks; i += 2) {
    const int c = nchunks - 1 - i;
    step(c, i, Xb0, Yb0, Cb0, Xb1, Yb1, Cb1);
    if (c > 0) {
      if (Cfg::NBUF == 2) step(c - 1, i + 1, Xb1, Yb1, Cb1, Xb0, Yb0, Cb0);
      else step(c - 1, i + 1, Xb0, Yb0, Cb0, Xb0, Yb0, Cb0);
    }
  }
}

// ------------------------------------------------------------- rows sweep

// Row layout (lane = column p), as in the forward: with 8 modes the columns of P
// are split over two workgroups; the 8 waves are NPW blocks of 16 columns times
// NPART parts splitting the modes (or N, with one mode).
template <typename T, int MP, int NB>
struct RowCfg {
  static constexpr int NP = NB * 16;
  static constexpr bool kBf16 = sizeof(T) == 2;
  static constexpr int XS = Pad<T>::XS;
  static constexpr int BS = Pad<T>::template CS<NP>;  // B read along rows (readout A operand)
  static constexpr int CS = Pad<T>::template BS<NP>;  // C read transposed (update A operand)
  static constexpr int NBUF = kBf16 ? 2 : 1;
  // (float32 tiles take twice the LDS: no P split there, the exchange would not fit)
  static constexpr int PS = (MP >= 8 && kBf16) ? 2 : 1;
  static constexpr int NPW = 4 / PS;
  static constexpr bool kModeSplit = MP >= 2;
  static constexpr int NPART = kModeSplit ? 8 / NPW : (NB >= 2 ? 2 : 1);
  static constexpr int MPW = kModeSplit ? MP / NPART : MP;
  static constexpr int NBW = (!kModeSplit && NB >= 2) ? NB / 2 : NB;
  static constexpr int KBW = (NBW + 1) / 2;
  static constexpr int TBP = (kBf16 ? MPW * NBW < 16 : MPW * NBW < 8) ? 4 : (kBf16 || MPW * NBW < 16) ? 2 : 1;
};

template <typename T, int MP, int NB>
__global__ void __launch_bounds__(512) frac_bwd_rows_kernel(ScanParams p, BwdWork wk) {
  using Cfg = RowCfg<T, MP, NB>;
  constexpr int NP = Cfg::NP, XS = Cfg::XS, BS = Cfg::BS, CS = Cfg::CS;
  constexpr int NPART = Cfg::NPART, MPW = Cfg::MPW, NBW = Cfg::NBW, KBW = Cfg::KBW, TBP = Cfg::TBP;
  using Ex = Exchange<NPART>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M, G = p.G;
  const int nchunks = (L + kQ - 1) / kQ;
  int b, h, ps;
  block_head(Cfg::PS, H, b, h, ps);
  const int g = h * G / H;
  const int pbl = wave % Cfg::NPW, part = wave / Cfg::NPW;
  const int pb = ps * Cfg::NPW + pbl;
  const bool active = pb * 16 < p.PP && part < NPART;
  const int mo = Cfg::kModeSplit ? part * MPW : 0;
  const int nbo = (!Cfg::kModeSplit && NPART == 2) ? part * NBW : 0;
  const int pc = pb * 16 + li;

  // B and x are needed early in a chunk only: single buffers refilled mid-chunk
  __shared__ __align__(16) T Bb[64 * BS], Xb[64 * XS];
  __shared__ __align__(16) T Cb0[64 * CS], Yb0[64 * XS];
  __shared__ __align__(16) T Cb1[Cfg::NBUF == 2 ? 64 * CS : 8], Yb1[Cfg::NBUF == 2 ? 64 * XS : 8];
  constexpr int NWA = n_weight_arrays<kRows>();
  constexpr int oGG = 0;                                         // T [t'][k] (C B^T) o Gamma, causal
  constexpr int oDx = oGG + 64 * XS * (int)sizeof(T);            // T [t][p] dx rows of the previous chunk (bf16)
  constexpr int oW = oDx + (Cfg::kBf16 ? 64 * XS * (int)sizeof(T) : 0);
  constexpr int oRd = oW + (NWA * MP * kWQ + kQ) * 4;             // float [2][8][Q] token partials of e, f
  constexpr int oEx = oRd + 2 * 8 * kQ * 4;
  constexpr int oSc = oEx + Ex::kFloats * 4;
  __shared__ __align__(16) unsigned char sm[oSc + 4 * MP * 4];
  T* GG = reinterpret_cast<T*>(sm + oGG);
  T* Dxb = reinterpret_cast<T*>(sm + oDx);
  float* W = reinterpret_cast<float*>(sm + oW);
  float* P_A = W + NWA * MP * kWQ;
  float* redE = reinterpret_cast<float*>(sm + oRd);
  float* redF = redE + 8 * kQ;
  float* XCH = reinterpret_cast<float*>(sm + oEx);
  float* s_rr = reinterpret_cast<float*>(sm + oSc);
  float* s_lnt = s_rr + MP;
  float* s_E2 = s_lnt + MP;
  constexpr int SW = MP * kWQ;  // stride of the weight arrays
  const float* P_wdx = W;  // times r_m: the adjoint weight of e
  const float* P_wfk = W + 1 * SW;
  const float* P_om = W + 2 * SW;

  if (tid < MP) {
    const float tau = (tid < M) ? p.tau[tid] : 1.0f;
    s_rr[tid] = (tid < M) ? 1.0f / tau : 0.0f;
    s_lnt[tid] = (tid < M) ? logf(tau) : 0.0f;
    s_E2[tid] = 1.0f;
  }
  for (int i = tid; i < 64 * XS; i += 512) {
    GG[i] = (T)0.0f;
    Xb[i] = Yb0[i] = (T)0.0f;
    Yb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;
  }
  for (int i = tid; i < 64 * BS; i += 512) Bb[i] = (T)0.0f;
  for (int i = tid; i < 64 * CS; i += 512) Cb0[i] = Cb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;

  // ---- adjoint G: Gs[m][jb] holds mode mo + m, rows n = 16 (nbo + jb) + 4 lg + r, column pc
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)M * N * P;
  floatx4 Gs[MPW][NBW];
  {
    int lo = (mo * N + nbo * 16 + lg * 4) * P + pc;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MPW; ++m)
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = (nbo + jb) * 16 + lg * 4 + r;
          float v = 0.0f;
          if (p.d_final_state && active && mo + m < M && n < N && pc < P)
            v = p.d_final_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * P];
          Gs[m][jb][r] = v;
        }
  }
  const float Dh = p.D ? p.D[h] : 0.0f;

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * P;
  const T* yg = reinterpret_cast<const T*>(p.dy) + (((int64_t)b * L) * H + h) * P;
  T* dxg = reinterpret_cast<T*>(p.dx) + (((int64_t)b * L) * H + h) * P;
  const T* Bgp = reinterpret_cast<const T*>(p.Bm) + (((int64_t)b * L) * G + g) * N;
  const T* Cgp = reinterpret_cast<const T*>(p.Cm) + (((int64_t)b * L) * G + g) * N;
  const int64_t xstride = (int64_t)H * P, bstride = (int64_t)G * N;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const int64_t lg_st = (int64_t)H * M;
  PairLogits<MP, 512> lgt_n;  // the logits of the next chunk's weight pass
  auto load_controls = [&](int c, float& dtv, float& al, float& lam) {
    const int tg = c * kQ + lane;
    const bool valid = tg < L;
    dtv = valid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al = valid ? al_bh[tg * p.as1] : 1.0f;
    lam = (valid && lm_bh) ? lm_bh[tg * p.ls1] : 1.0f;
    lgt_n.load(rl_bh, wl_bh, c * kQ, min(kQ, L - c * kQ), M, lg_st, threadIdx.x);
  };
  DmaPlan<T, XS> planX;
  DmaPlan<T, BS> planB;
  DmaPlan<T, CS> planC;
  planX.init(xstride, P);
  planB.init(bstride, N);
  planC.init(bstride, N);
  auto stage_late = [&](int c, T* Cd, T* Yd) {  // used through the whole chunk
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    planC.issue_async(Cd, Cgp + (int64_t)t0 * bstride, bstride, nv);
    planX.issue_async(Yd, yg + (int64_t)t0 * xstride, xstride, nv);
  };
  auto stage_early = [&](int c) {  // read before the mid-chunk barrier only
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    planB.issue_async(Bb, Bgp + (int64_t)t0 * bstride, bstride, nv);
    planX.issue_async(Xb, xg + (int64_t)t0 * xstride, xstride, nv);
  };
  // dx rows of chunk c (staged in Dxb) -> global, this workgroup's columns
  auto store_dx = [&](int c) {
    constexpr int E8 = 16 / sizeof(T);
    constexpr int CY = 64 / E8;
    const int t0 = c * kQ, nv = min(kQ, L - t0);
#pragma unroll
    for (int i0 = 0; i0 < 64 * CY; i0 += 512) {
      const int i = i0 + tid, t = i / CY, ch = i & (CY - 1);
      const int col = ch * E8;
      if (t < nv && col < P && col >= ps * Cfg::NPW * 16 && col < (ps + 1) * Cfg::NPW * 16)
        *reinterpret_cast<int4*>(dxg + (int64_t)(t0 + t) * xstride + col) =
            *reinterpret_cast<const int4*>(Dxb + t * XS + col);
    }
  };

  float dt_n, al_n, lam_n;
  load_controls(nchunks - 1, dt_n, al_n, lam_n);
  if (Cfg::NBUF == 2) {
    stage_late(nchunks - 1, Cb0, Yb0);
    stage_early(nchunks - 1);
  }
  // (C B^T) o Gamma tiles written by the state sweep, loaded one chunk ahead (in processing order)
  const T* ggtiles = reinterpret_cast<const T*>(wk.gg);
  const int64_t bl_h = (int64_t)p.Bsz * L * H;
  TilePrefetch<T> ggt;
  ggt.load(ggtiles + ((int64_t)(b * nchunks + nchunks - 1) * H + h) * (kTiles * kTileElems), wave, lane);

  auto step = [&](int c, int i, T* Cc, T* Yc, T* Cn, T* Yn) __attribute__((always_inline)) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    const float* Ecur = s_E2 + (i & 1) * MP;
    float* Enext = s_E2 + ((i + 1) & 1) * MP;
    wait_vmem();
    barrier();
    // this chunk's prefetched controls, logits and tile values, taken before any new memory operation
    const float dtv = pinned(dt_n), al_l = pinned(al_n), lam_l = pinned(lam_n);
    const PairLogits<MP, 512> lgt = lgt_n.pinned_copy();
    const TilePrefetch<T> gcur = ggt.pinned_copy();
    if (Cfg::kBf16 && i > 0) store_dx(c + 1);
    if (Cfg::NBUF == 2) {
      if (c > 0) stage_late(c - 1, Cn, Yn);
    } else {
      stage_late(c, Cc, Yc);
      stage_early(c);
      wait_vmem();
      barrier();
    }
    if (c > 0) load_controls(c - 1, dt_n, al_n, lam_n);
    const ChunkCtl k = chunk_controls(dtv, al_l, lam_l, lm_bh != nullptr, nv);
    if (wave == 0) P_A[lane] = k.A;
    const int unsafe = pair_weights<MP, kRows>(k, nv, M, lgt, rl_bh == wl_bh, s_rr, s_lnt, Ecur, Enext, W);
    float renf[MPW];
    int renbits = 0;
#pragma unroll
    for (int m = 0; m < MPW; ++m) {
      const float Enew = uniform(Ecur[mo + m] * fexp(-s_rr[mo + m] * k.Alast));
      renf[m] = Enew;
      if (__float_as_int(Enew) < __float_as_int(kRescaleFloor)) renbits |= 1 << m;
    }
    barrier();  // weights in LDS

    __builtin_amdgcn_sched_barrier(0);
    // ---- GG = (C B^T) o Gamma, natural [t'][k], causal (tiles from the state sweep)
    {
#pragma unroll
      for (int jt = 0; jt < 2; ++jt) {
        const int tile = wave + 8 * jt;
        if (tile >= kTiles) break;
        const int tb = tile_row(tile), kb = tile_col(tile);
#pragma unroll
        for (int r = 0; r < 4; ++r) GG[(tb * 16 + lg * 4 + r) * XS + kb * 16 + li] = gcur.v[jt].e[r];
      }
    }
    (void)unsafe;

    if (c > 0) ggt.load(ggtiles + ((int64_t)(b * nchunks + c - 1) * H + h) * (kTiles * kTileElems), wave, lane);

    __builtin_amdgcn_sched_barrier(0);
    // ---- Z^T_m = G_m^T B^T (rows p of this wave's block, columns t) -> dx^T (inter)
    // and the adjoint parts of e, f
    floatx4 dxa[4];  // dx^T: rows p = 16 pb + 4 lg + r, column t = 16 tb + li
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) dxa[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    {
      float ekf[4] = {0.f, 0.f, 0.f, 0.f}, fkf[4] = {0.f, 0.f, 0.f, 0.f};  // this lane's token, per row block
      if (active) {
#pragma unroll
        for (int tp = 0; tp < 4 / TBP; ++tp) {
          Frag<T> Ba[TBP][KBW];
#pragma unroll
          for (int q = 0; q < TBP; ++q)
#pragma unroll
            for (int kb = 0; kb < KBW; ++kb) {
              const T* row = Bb + ((tp * TBP + q) * 16 + li) * BS + nbo * 16 + kb * 32 + lg * 4;
              Ba[q][kb] = frag_load4x2(row, row + 16, 2 * kb + 1 < NBW);
            }
          floatx4 We[TBP], Wf[TBP];
#pragma unroll
          for (int q = 0; q < TBP; ++q) We[q] = Wf[q] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int m = 0; m < MPW; ++m) {
            Frag<T> Gf[KBW];
#pragma unroll
            for (int kb = 0; kb < KBW; ++kb) {
#pragma unroll
              for (int s = 0; s < 4; ++s) frag_set(Gf[kb], s, Gs[m][2 * kb][s]);
#pragma unroll
              for (int s = 0; s < 4; ++s) frag_set(Gf[kb], 4 + s, (2 * kb + 1 < NBW) ? Gs[m][2 * kb + 1][s] : 0.0f);
            }
            const float rm = s_rr[mo + m];
#pragma unroll
            for (int q = 0; q < TBP; ++q) {
              const int tb = tp * TBP + q;
              floatx4 Z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
              for (int kb = 0; kb < KBW; ++kb) mma(Z, Gf[kb], Ba[q][kb]);
              const int o = (mo + m) * kWQ + tb * 16 + li;
              const float wx = P_wdx[o], wf = P_wfk[o], rwx = rm * wx;
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                dxa[tb][r] = __builtin_fmaf(wx, Z[r], dxa[tb][r]);
                We[q][r] = __builtin_fmaf(rwx, Z[r], We[q][r]);
                Wf[q][r] = __builtin_fmaf(wf, Z[r], Wf[q][r]);
              }
            }
          }
#pragma unroll
          for (int q = 0; q < TBP; ++q) {
            const int tb = tp * TBP + q;
            float xv[4];
            load4(Xb + (tb * 16 + li) * XS + pb * 16 + lg * 4, xv);
            ekf[tb] = We[q][0] * xv[0] + We[q][1] * xv[1] + We[q][2] * xv[2] + We[q][3] * xv[3];
            fkf[tb] = Wf[q][0] * xv[0] + Wf[q][1] * xv[1] + Wf[q][2] * xv[2] + Wf[q][3] * xv[3];
          }
        }
        if (NPART > 1) Ex::put(XCH, wave, part, dxa);
      }
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        float e = ekf[tb], f = fkf[tb];
        e = xor32_sum(xor16_sum(e));
        f = xor32_sum(xor16_sum(f));
        if (lg == 0) {
          redE[wave * kQ + tb * 16 + li] = e;
          redF[wave * kQ + tb * 16 + li] = f;
        }
      }
    }
    barrier();  // GG, exchange and token partials complete; B and x are free
    if (Cfg::NBUF == 2 && c > 0) stage_early(c - 1);

    if (wave == 0) {
      const int t = lane;
      float e = 0.f, f = 0.f;
      for (int w2 = 0; w2 < 8; ++w2) {
        e += redE[w2 * kQ + t];
        f += redF[w2 * kQ + t];
      }
      if (t < nv) {
        const int64_t ith = ((int64_t)b * H + h) * L + t0 + t;  // [B, H, L]
        wk.eB[ps * bl_h + ith] = e;
        wk.fB[ps * bl_h + ith] = f;
      }
    }
    if (!active) return;

    __builtin_amdgcn_sched_barrier(0);
    // ---- dx^T blocks this wave finishes: other parts + intra dY^T GG (t' >= t) + D dy
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      if (!Ex::owns(tb, part)) continue;
      if (NPART > 1) Ex::gather(XCH, part, tb, dxa[tb], [&](int q) { return q * Cfg::NPW + pbl; });
#pragma unroll
      for (int kk = tb / 2; kk < 2; ++kk) {
        const Frag<T> a = frag_load_rows(Yc, XS, kk * 32 + lg * 8, pb * 16);
        const Frag<T> bb = frag_load_rows(GG, XS, kk * 32 + lg * 8, tb * 16);
        mma(dxa[tb], a, bb);
      }
      const int t = tb * 16 + li, pr = pb * 16 + lg * 4;
      float yv[4];
      load4(Yc + t * XS + pr, yv);
      floatx4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = dxa[tb][r] + Dh * yv[r];
      if (Cfg::kBf16) store4(Dxb + t * XS + pr, v);  // staged, stored 16 bytes at a time
      else if (t < nv && pr < P) store4(dxg + (int64_t)t0 * xstride + t * (H * P) + pr, v);
    }

    __builtin_amdgcn_sched_barrier(0);
    // ---- adjoint update G += C^T (omega o dY), rows n, column pc
#pragma unroll
    for (int m = 0; m < MPW; ++m) {
      if (!((renbits >> m) & 1)) continue;
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) Gs[m][jb][r] *= renf[m];
    }
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const Frag<T> yf = frag_load_rows(Yc, XS, kt * 32 + lg * 8, pb * 16);
      Frag<T> Yf[MPW];
#pragma unroll
      for (int m = 0; m < MPW; ++m) {
        const float* pv = P_om + (mo + m) * kWQ + kt * 32 + lg * 8;
        const float4 v0 = *reinterpret_cast<const float4*>(pv);
        const float4 v1 = *reinterpret_cast<const float4*>(pv + 4);
        frag_set(Yf[m], 0, to_f32(yf.v[0]) * v0.x);
        frag_set(Yf[m], 1, to_f32(yf.v[1]) * v0.y);
        frag_set(Yf[m], 2, to_f32(yf.v[2]) * v0.z);
        frag_set(Yf[m], 3, to_f32(yf.v[3]) * v0.w);
        frag_set(Yf[m], 4, to_f32(yf.v[4]) * v1.x);
        frag_set(Yf[m], 5, to_f32(yf.v[5]) * v1.y);
        frag_set(Yf[m], 6, to_f32(yf.v[6]) * v1.z);
        frag_set(Yf[m], 7, to_f32(yf.v[7]) * v1.w);
      }
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb) {
        const Frag<T> a = frag_load_rows(Cc, CS, kt * 32 + lg * 8, (nbo + jb) * 16);
#pragma unroll
        for (int m = 0; m < MPW; ++m) mma(Gs[m][jb], a, Yf[m]);  // modes >= M carry zero weights
      }
    }
  };

  for (int i = 0; i < nchunks; i += 2) {
    const int c = nchunks - 1 - i;
    step(c, i, Cb0, Yb0, Cb1, Yb1);
    if (c > 0) {
      if (Cfg::NBUF == 2) step(c - 1, i + 1, Cb1, Yb1, Cb0, Yb0);
      else step(c - 1, i + 1, Cb0, Yb0, Cb0, Yb0);
    }
  }
  wait_vmem();
  barrier();
  if (Cfg::kBf16) store_dx(0);
}

// ---------------------------------------------------------- finishing kernels

// ddt from the per-token terms: suffix sums over the sequence, in two steps with
// a fixed summation order.  First the total of e over each 64-token tile of each
// (batch, head); then one block of 16 waves per (batch, tile, 64 heads) forms, per head, the
// sum over the later tiles, the suffix sums inside the tile (one wave per head,
// lane = token), and writes ddt through LDS so that each token's heads are stored
// contiguously.

// e_t of one token: readout / intra parts minus adjoint parts (partials per half).
__device__ __forceinline__ float ddt_e(const BwdWork& wk, int64_t blh, int64_t i, int nA, int nB) {
  float e = 0.0f;
  for (int q = 0; q < nA; ++q) e += wk.eA[q * blh + i];
  for (int q = 0; q < nB; ++q) e -= wk.eB[q * blh + i];
  return e;
}

__global__ void __launch_bounds__(256) frac_bwd_ddt_tiles_kernel(ScanParams p, BwdWork wk, float* tsum, int nA,
                                                                 int nB) {
  const int ntiles = (p.L + 63) / 64;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (b h) * ntiles + tile
  const int lane = threadIdx.x & 63;
  if (wid >= (int64_t)p.Bsz * p.H * ntiles) return;
  const int64_t bh = wid / ntiles;
  const int t = (int)(wid - bh * ntiles) * 64 + lane;
  const int64_t blh = (int64_t)p.Bsz * p.L * p.H;
  float e = t < p.L ? ddt_e(wk, blh, bh * p.L + t, nA, nB) : 0.0f;
  e = group_allreduce<64>(e, [](float x, float y) { return x + y; });
  if (lane == 0) tsum[wid] = e;
}

__global__ void __launch_bounds__(1024) frac_bwd_ddt_kernel(ScanParams p, BwdWork wk, const float* tsum, int nA,
                                                           int nB, int nD) {
  __shared__ float carry[64];
  __shared__ float out[64][65];
  const int L = p.L, H = p.H, ntiles = (L + 63) / 64;
  const int b = blockIdx.x / ntiles, tile = blockIdx.x - b * ntiles, h0 = blockIdx.y * 64, t0 = tile * 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nh = min(64, H - h0);
  const int64_t blh = (int64_t)p.Bsz * L * H, bhn = (int64_t)p.Bsz * H;
  // per head: final-state term plus the totals of e over the later tiles (one wave
  // per head, lane j adding tiles tile + 1 + j, tile + 65 + j, ...)
  for (int hl = wave; hl < nh; hl += 16) {
    const int64_t bh = (int64_t)b * H + h0 + hl;
    float later = 0.0f;
    for (int j = tile + 1 + lane; j < ntiles; j += 64) later += tsum[bh * ntiles + j];
    later = group_allreduce<64>(later, [](float x, float y) { return x + y; });
    if (lane == 0) {
      float Fv = 0.0f;
      for (int q = 0; q < nA; ++q) Fv += wk.F[q * bhn + bh];
      carry[hl] = Fv + later;
    }
  }
  __syncthreads();
  const int t = t0 + lane;
  for (int hl = wave; hl < nh; hl += 16) {
    const int h = h0 + hl;
    const int64_t i = ((int64_t)b * H + h) * L + t;  // [B, H, L]
    float e = 0.0f, f = 0.0f;
    if (t < L) {
      e = ddt_e(wk, blh, i, nA, nB);
      for (int q = 0; q < nA; ++q) f += wk.fA[q * blh + i];
      for (int q = 0; q < nB; ++q) f += wk.fB[q * blh + i];
    }
    // inclusive suffix sum over the tile: within each 16-lane row (lanes above,
    // zero past the row end), then the totals of the later rows
    float s = e;
    s += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(s), 0x101, 0xF, 0xF, true));  // row_shl:1
    s += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(s), 0x102, 0xF, 0xF, true));  // row_shl:2
    s += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(s), 0x104, 0xF, 0xF, true));  // row_shl:4
    s += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(s), 0x108, 0xF, 0xF, true));  // row_shl:8
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), 48));
    const int row = lane >> 4;
    const float rows_after = row == 0 ? (r3 + r2) + r1 : row == 1 ? r3 + r2 : row == 2 ? r3 : 0.0f;
    s += rows_after;
    float v = 0.0f;
    if (t < L) {
      const float al = strided3(p.alpha, p.as0, p.as1, p.as2, b, t, h);
      const float lam = p.lambda ? strided3(p.lambda, p.ls0, p.ls1, p.ls2, b, t, h) : 1.0f;
      const float s_eff = p.lambda ? step_factor(lam, al) : 1.0f;
      v = (-carry[hl] - s + f) * s_eff;
    }
    out[lane][hl] = v;
  }
  __syncthreads();
  for (int k = tid; k < 64 * 64; k += 1024) {
    const int tt = k >> 6, hl = k & 63;
    if (t0 + tt < L && hl < nh) p.ddt[((int64_t)b * L + t0 + tt) * H + h0 + hl] = out[tt][hl];
  }
  if (p.dD && b == 0 && tile == 0 && tid < nh) {
    float acc = 0.0f;
    for (int q = 0; q < nD; ++q)
      for (int bb = 0; bb < p.Bsz; ++bb) acc += wk.dDp[((int64_t)q * p.Bsz + bb) * H + h0 + tid];
    p.dD[h0 + tid] = acc;
  }
}

// dB, dC of each group: fixed-order sum of the per-head partials; each thread
// sums 16 bytes of a (token, group) row over the group's heads.
template <typename T>
__global__ void __launch_bounds__(256) frac_bwd_group_sum_kernel(ScanParams p, const T* __restrict__ dBp,
                                                                 const T* __restrict__ dCp, int64_t nrows) {
  constexpr int E = 16 / sizeof(T);
  const int H = p.H, N = p.N, G = p.G, hpg = H / G, cpr = N / E;  // 16-byte chunks per row
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= nrows * G * cpr) return;
  const int ch = (int)(i % cpr);
  const int64_t rg = i / cpr;  // (b * L + t) * G + g
  const int g = (int)(rg % G);
  const int64_t bt = rg / G;
  float sb[E], sc[E];
#pragma unroll
  for (int k = 0; k < E; ++k) sb[k] = sc[k] = 0.0f;
  for (int j = 0; j < hpg; ++j) {
    const int64_t off = (bt * H + g * hpg + j) * N + ch * E;
    float vb[E], vc[E];
    if constexpr (E == 8) {
      load8(dBp + off, vb);
      load8(dCp + off, vc);
    } else {
      load4(dBp + off, vb);
      load4(dCp + off, vc);
    }
#pragma unroll
    for (int k = 0; k < E; ++k) {
      sb[k] += vb[k];
      sc[k] += vc[k];
    }
  }
  T* dB = reinterpret_cast<T*>(p.dBm) + rg * N + ch * E;
  T* dC = reinterpret_cast<T*>(p.dCm) + rg * N + ch * E;
#pragma unroll
  for (int k = 0; k < E; ++k) {
    dB[k] = (T)sb[k];
    dC[k] = (T)sc[k];
  }
}

struct BwdLayout {
  size_t tiles, gg, hg, dBp, dCp, scal, total;
};

BwdLayout bwd_layout(const ScanParams& p) {
  BwdLayout l{};
  const size_t es = p.io_bf16 ? 2 : 4;
  const size_t bl = (size_t)p.Bsz * p.L;
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  l.tiles = 0;
  const size_t gtb = (size_t)p.Bsz * ((p.L + kQ - 1) / kQ) * p.H * kTiles * kTileElems * es;
  l.gg = up(cb_tiles_bytes(p));
  l.hg = l.gg + up(gtb);
  l.dBp = l.hg + up(gtb);
  l.dCp = l.dBp + up(bl * p.H * p.N * es);
  l.scal = l.dCp + up(bl * p.H * p.N * es);
  // eA[2], fA[2], eB[2], fB[2] per token and head; F[2], dDp per head; tile totals
  l.total = l.scal + up(sizeof(float) * (8 * bl * p.H + 3 * (size_t)p.Bsz * p.H +
                                         (size_t)p.Bsz * p.H * ((p.L + 63) / 64)));
  return l;
}

template <typename T, int MP, int NB>
hipError_t launch_bwd_variant(const ScanParams& p, void* ws, hipStream_t stream) {
  const BwdLayout l = bwd_layout(p);
  unsigned char* base = reinterpret_cast<unsigned char*>(ws);
  BwdWork wk;
  wk.tiles = base + l.tiles;
  wk.gg = base + l.gg;
  wk.hg = base + l.hg;
  wk.dBp = base + l.dBp;
  wk.dCp = base + l.dCp;
  float* sc = reinterpret_cast<float*>(base + l.scal);
  const size_t blh = (size_t)p.Bsz * p.L * p.H;
  wk.eA = sc;
  wk.fA = sc + 2 * blh;
  wk.eB = sc + 4 * blh;
  wk.fB = sc + 6 * blh;
  wk.F = sc + 8 * blh;
  wk.dDp = wk.F + 2 * (size_t)p.Bsz * p.H;
  wk.tsum = wk.dDp + (size_t)p.Bsz * p.H;

  hipError_t e = launch_cb_tiles(p, base + l.tiles, stream);
  if (e != hipSuccess) return e;
  const int bh = p.Bsz * p.H;
  hipLaunchKernelGGL((frac_bwd_state_kernel<T, MP, NB>), dim3(bh * ColCfg<T, MP, NB>::PS), dim3(512), 0, stream, p,
                     wk);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((frac_bwd_rows_kernel<T, MP, NB>), dim3(bh * RowCfg<T, MP, NB>::PS), dim3(512), 0, stream, p,
                     wk);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((frac_bwd_cols_kernel<T, MP, NB>), dim3(bh * ColCfg<T, MP, NB>::PS), dim3(512), 0, stream, p,
                     wk);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  {
    const int ntiles = (p.L + 63) / 64;
    const int64_t nt = (int64_t)bh * ntiles;
    hipLaunchKernelGGL(frac_bwd_ddt_tiles_kernel, dim3((unsigned)((nt + 3) / 4)), dim3(256), 0, stream, p, wk, wk.tsum,
                       ColCfg<T, MP, NB>::PS, RowCfg<T, MP, NB>::PS);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(frac_bwd_ddt_kernel, dim3((unsigned)(ntiles * p.Bsz), (p.H + 63) / 64), dim3(1024), 0, stream, p, wk,
                       (const float*)wk.tsum, ColCfg<T, MP, NB>::PS, RowCfg<T, MP, NB>::PS, 1);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t nrows = (int64_t)p.Bsz * p.L;
  const int64_t nthr = nrows * p.G * (p.N / (16 / (int)sizeof(T)));
  hipLaunchKernelGGL((frac_bwd_group_sum_kernel<T>), dim3((unsigned)((nthr + 255) / 256)), dim3(256), 0, stream, p,
                     reinterpret_cast<const T*>(wk.dBp), reinterpret_cast<const T*>(wk.dCp), nrows);
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

hipError_t launch_ddt_finish(const ScanParams& p, float* eA, float* fA, float* eB, float* fB, float* F, float* dDp,
                             float* tsum, int nA, int nB, int nD, hipStream_t stream) {
  BwdWork wk{};
  wk.eA = eA;
  wk.fA = fA;
  wk.eB = eB;
  wk.fB = fB;
  wk.F = F;
  wk.dDp = dDp;
  wk.tsum = tsum;
  const int ntiles = (p.L + 63) / 64;
  const int64_t nt = (int64_t)p.Bsz * p.H * ntiles;
  hipLaunchKernelGGL(frac_bwd_ddt_tiles_kernel, dim3((unsigned)((nt + 3) / 4)), dim3(256), 0, stream, p, wk, tsum, nA,
                     nB);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(frac_bwd_ddt_kernel, dim3((unsigned)(ntiles * p.Bsz), (p.H + 63) / 64), dim3(1024), 0, stream, p,
                     wk, (const float*)tsum, nA, nB, nD);
  return hipGetLastError();
}

size_t scan_bwd_workspace(const ScanParams& p) {
  if (p.Bsz == 0 || p.L == 0) return 0;
  return bwd_layout(p).total;
}

hipError_t launch_scan_bwd(const ScanParams& p, void* ws, size_t, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  return p.io_bf16 ? launch_bwd_mp<bf16>(p, ws, stream) : launch_bwd_mp<float>(p, ws, stream);
}

}  // namespace frac
