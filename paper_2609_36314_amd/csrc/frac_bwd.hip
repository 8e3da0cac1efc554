// frac_bwd.hip -- chunked parallel scan, backward (training).
//
// Reverse-mode derivative of the selective mode-bank recurrence of Sec. 3.2
// (eq. frac-selective-update, eq. frac-readout, the Appendix-D algorithm), with
// the B/C-widened state, evaluated chunk by chunk like the forward.  Per mode,
// chunk log-decays l (the chunk-local sums of the capped exponents r_m dtt, in
// float64), chunk total l_Q, state entering the chunk S0 and adjoint of the
// chunk's last state G:
//
//   dC_t  = sum_m c_{t,m} e^{-l_t} S0_m dy_t + sum_{k<=t} Gamma_{t,k} (dy_t . x_k) B_k
//   dx_t  = sum_m kappa_{t,m} e^{-(l_Q - l_t)} B_t G_m
//           + sum_{t'>=t} Gamma_{t',t} (C_t' . B_t) dy_t' + D dy_t
//   dB_t  = sum_m kappa_{t,m} e^{-(l_Q - l_t)} G_m x_t
//           + sum_{t'>=t} Gamma_{t',t} (dy_t' . x_t) C_t'
//   G (entering the previous chunk) = e^{-l_Q} G + sum_t c_{t,m} e^{-l_t} C_t dy_t^T
//
// and the gradients of the per-(token, mode) weights, from which the finishing
// kernels (frac_grads.hip) form ddt, dalpha, dlambda and the logit gradients:
//   dc_{t,m} = e^{-l_t} C_t . (S0_m dy_t) + sum_{k<=t} H_{t,k} kappa_{k,m} e^{-(l_t - l_k)}
//   dk_{t,m} = e^{-(l_Q - l_t)} (B_t^T G_m) . x_t + sum_{t'>=t} H_{t',t} c_{t',m} e^{-(l_t' - l_t)}
//   H = (C B^T) o (dY X^T)
//
// Three sweeps, each its own kernel; every wave keeps its share of a state or
// adjoint (at most 2 x 4 16x16 float32 tiles per mode group) in matrix-core
// accumulators for the whole sequence:
//   state  forward in time, state transposed (lane = column n of N, rows p): dC
//          (per head), dc (per mode, over the workgroup's rows of N; with the
//          intra-chunk parts of dc and dk when they fit in LDS), the final-state
//          term <dS_final, S_final> per mode and sum(dy . x) for dD;
//   rows   reverse, adjoint in row layout (lane = column p of P, rows n): dx, the
//          inter-chunk part of dk (through the adjoint carried in from the later
//          chunks, per mode, over the workgroup's columns of P), the gradient of
//          the initial state and the term <S_init, dS_init> per mode;
//   cols   reverse, adjoint transposed (lane = column n): dB (per head).
// The state sweep also writes each chunk's causal tiles (C B^T) o Gamma and
// Gamma o (dY X^T) (bfloat16 for bfloat16 I/O, 10 tiles of 16x16 per chunk and
// head), which the reverse sweeps read instead of forming Gamma again.  With many
// modes and a wide state the state and cols sweeps split N, and the rows sweep
// splits P, over two workgroups per (batch, head), so that no per-head output
// gets a second partial sum.  Tiles are copied straight into
// LDS (natural layout, padded rows) and read back as matrix-core fragments with
// row reads or transposed 64-bit reads.  A chunk-parallel kernel forms the
// intra-chunk parts of dc and dk where the state sweep cannot, the finisher of
// frac_grads.hip turns the per-(token, mode) partials into the step-size, order
// and logit gradients, and a reduction kernel sums dB and dC over the heads of
// each group in a fixed order.  Banks of more than eight modes run the sweeps once
// per block of eight modes, and heads wider than 64 columns once per group of 64
// columns, each with slots of its own for the sums that span them.
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
enum Role { kState = 0, kRows = 1, kCols = 2, kIntra = 3 };

// Number of [MP][Q] weight arrays a role keeps in LDS (plus two for the hi and lo
// parts of the chunk log-decays).
template <int ROLE>
constexpr int n_weight_arrays() {
  return ROLE == kState ? 4 : ROLE == kRows ? 3 : 2;
}

// Per-wave chunk controls (lane = token): the effective step and the fractional order.
struct ChunkCtl {
  float dtt, al;
};

__device__ __forceinline__ ChunkCtl chunk_controls(float dtv, float al, float lam, bool has_lambda, int nv) {
  const int lane = threadIdx.x & 63;
  ChunkCtl k;
  const float s_eff = has_lambda ? step_factor(lam, al) : 1.0f;
  k.dtt = (lane < nv) ? dtv * s_eff : 0.0f;
  k.al = al;
  return k;
}

// Per-(token, mode) weights of one chunk, pair = t * MP + m, written to the
// role's LDS arrays w[i * MP * Q + m * Q + t], from the chunk log-decays l (hi and
// lo parts lh, ll).  Returns the modes whose chunk decay exceeds the factorisation
// bound (bit m); for those the Gamma arrays hold c and kappa without the exponentials.
//   state: 0 c e^{-l} (c), 1 kappa e^{l} (kappa), 2 c e^{-l} E, 3 kappa e^{-(l_Q-l)} upd
//   rows:  0 kappa e^{-(l_Q-l)} E, 1 e^{-(l_Q-l)} E, 2 c e^{-l} upd
//   cols:  0 kappa e^{-(l_Q-l)} E, 1 c e^{-l} upd
//   intra: 0 c e^{-l} (c), 1 kappa e^{l} (kappa)
// (the reverse sweeps read their Gamma tiles from the state sweep)
// E is the scale of the state (or adjoint) before this chunk's update, upd the
// factor on the update (1/E_new, or 1 when the accumulators are folded back).
// BLK (one block of a mode-block launch sequence): the weights are normalised over
// the whole bank with the per-token log-normalizers that lgt carries (lane = token).
template <int MP, int ROLE, int NT = 512, bool BLK = false>
__device__ __forceinline__ int pair_weights(const ChunkCtl& k, int nv, int M, const PairLogits<MP, NT, BLK>& lgt,
                                            bool w_is_c, const float* s_rr, const float* s_lnt, const float* lh,
                                            const float* ll, const float* Ecur, float* Enext, float* w) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int j = 0; j < lgt.NPR; ++j) {
    const int pr = tid + NT * j;
    if (pr >= kQ * MP) break;  // wave-uniform
    const int t = pr / MP, m = pr - t * MP;
    const float dtt = __shfl(k.dtt, t, 64), al = __shfl(k.al, t, 64);
    const bool valid = t < nv;
    const float r = s_rr[m], prior = -al * s_lnt[m];
    const float zc = (m < M) ? prior + lgt.rl[j] : -INFINITY;
    const float zw = (m < M) ? prior + lgt.wl[j] : -INFINITY;
    // tokens past the sequence get zero weights (their tile rows may hold anything finite)
    float cw, ww;
    if constexpr (BLK) {
      const float lnc = __shfl(lgt.ln_c, t, 64), lnw = __shfl(lgt.ln_w, t, 64);
      cw = valid ? __expf(zc - lnc) : 0.0f;
      ww = w_is_c ? cw : (valid ? __expf(zw - lnw) : 0.0f);
    } else {
      cw = valid ? group_softmax<MP>(zc) : 0.0f;
      ww = w_is_c ? cw : (valid ? group_softmax<MP>(zw) : 0.0f);
    }
    const float lt = lh[m * kWQ + t], lQ = lh[m * kWQ + kQ - 1];
    const bool safe = lQ <= kSafeExponent;
    const float kap = one_minus_exp_neg(dtt * r) * ww;
    const float ea = fexp(-lt);
    float* o = w + m * kWQ + t;
    constexpr int SW = MP * kWQ;  // stride of the weight arrays
    if constexpr (ROLE == kState || ROLE == kIntra) {
      o[0 * SW] = safe ? cw * ea : cw;
      o[1 * SW] = safe ? kap * fexp(lt) : kap;
    }
    if constexpr (ROLE != kIntra) {
      const float E = Ecur[m];
      const float Enew = E * fexp(-lQ);
      const bool ren = !(Enew >= kRescaleFloor);
      const float upd = ren ? 1.0f : fast_rcp(Enew);
      const float dec = ell_decay(lh + m * kWQ, ll + m * kWQ, kQ - 1, t);
      if constexpr (ROLE == kState) {
        o[2 * SW] = cw * ea * E;
        o[3 * SW] = kap * dec * upd;
      } else if constexpr (ROLE == kRows) {
        o[0 * SW] = kap * dec * E;
        o[1 * SW] = dec * E;
        o[2 * SW] = cw * ea * upd;
      } else {
        o[0 * SW] = kap * dec * E;
        o[1 * SW] = cw * ea * upd;
      }
      if (pr < MP) Enext[m] = ren ? 1.0f : Enew;
    }
  }
  // the same flags in every wave: lane m < MP tests mode m
  const int lane = tid & 63;
  const bool over = lane < MP && lane < M && !(lh[(lane < MP ? lane : 0) * kWQ + kQ - 1] <= kSafeExponent);
  return (int)(__ballot(over) & ((MP >= 32) ? 0xffffffffull : ((1ull << MP) - 1)));
}

// Rank-M product sum_m a[m][row0 + i] b[m][col0 + j] over a 16x16 tile
// (float32 matrix cores, modes as K), in the accumulator layout, over the modes
// whose bit in `unsafe` is clear.
template <int MP>
__device__ __forceinline__ floatx4 rank_m_tile(const float* a, const float* bm, int row0, int col0, int unsafe,
                                               int tid = threadIdx.x) {
  const int li = tid & 15, lg = (tid >> 4) & 3;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < (MP + 3) / 4; ++q) {
    const int m = q * 4 + lg;
    const bool ok = m < MP && !((unsafe >> (m < MP ? m : 0)) & 1);
    const float av = (m < MP) ? a[(m < MP ? m : 0) * kWQ + row0 + li] : 0.0f;
    const float bv = (m < MP) ? bm[(m < MP ? m : 0) * kWQ + col0 + li] : 0.0f;
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(ok ? av : 0.0f, ok ? bv : 0.0f, acc, 0, 0, 0);
  }
  return acc;
}

// Modes past the factorisation bound: add the pairwise-decay terms of
// sum_m a_m[t] b_m[k] e^{-(l_{t,m} - l_{k,m})} (t >= k) to a 16x16 tile.
template <int MP>
__device__ __forceinline__ void unsafe_terms(floatx4& acc, int unsafe, const float* a, const float* bm,
                                             const float* lh, const float* ll, int tb, int kb, int tid = threadIdx.x) {
  const int li = tid & 15, lg = (tid >> 4) & 3;
  for (int m = 0; m < MP; ++m) {
    if (!((unsafe >> m) & 1)) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
      if (t >= k) acc[r] += a[m * kWQ + t] * bm[m * kWQ + k] * ell_decay(lh + m * kWQ, ll + m * kWQ, t, k);
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
  float* dc;          // [slots][B H L][M] partials of dL/dc: state sweep (per N part), then the intra kernel
  float* dk;          // [slots][B H L][M] partials of dL/dkappa: rows sweep (per P part), then the intra kernel
  float* F;           // [PS][B H][M] <dS_final, S_final> per mode (per N part)
  float* I;           // [PS_rows][B H][M] <S_init, dS_init> per mode (per P part of the rows sweep)
  float* dDp;         // [B H] sum(dy . x)
  float* dki;         // [B H L][M] the intra-chunk part of dL/dkappa (when the state sweep forms it)
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

// LDS of the state sweep (bytes): the staged tiles, the fixed arrays, one chunk's
// weights; and whether the intra-chunk products of dc and dk (the masked H tile in
// LDS) fit beside them (bfloat16 I/O).
template <typename T, int MP, int NB>
struct StateLds {
  using Cfg = ColCfg<T, MP, NB>;
  static constexpr int kTiles_ = (Cfg::NBUF * 64 * (2 * Cfg::XS + Cfg::BS) + 64 * Cfg::CS) * (int)sizeof(T);
  static constexpr int kFixed = 64 * Cfg::XS * (int)sizeof(T) +
                                (8 * Cfg::MPF * kQ + Exchange<Cfg::NACT>::kFloats + 4 * MP) * 4;
  static constexpr int WSZ = (n_weight_arrays<kState>() + 2) * MP * kWQ;  // floats
  static constexpr int kHH = 64 * Cfg::XS * (int)sizeof(T);
  static constexpr int kLimit = 160 * 1024 - 512;
  static constexpr bool kFold = sizeof(T) == 2 && kTiles_ + kFixed + kHH + WSZ * 4 <= kLimit;
  static constexpr int NWB = kTiles_ + kFixed + (kFold ? kHH : 0) + 2 * WSZ * 4 <= kLimit ? 2 : 1;
};

template <typename T, int MP, int NB, bool BLK = false>
__global__ void __launch_bounds__(512) frac_bwd_state_kernel(ScanParams p, BwdWork wk) {
  using Cfg = ColCfg<T, MP, NB>;
  constexpr int NP = Cfg::NP, XS = Cfg::XS, BS = Cfg::BS, CS = Cfg::CS;
  constexpr int NBF = Cfg::NBF, FPART = Cfg::FPART, MPF = Cfg::MPF;
  using Ex = Exchange<Cfg::NACT>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M, G = p.G;
  const int Ps = p.Pst;  // row stride of x, dy, dx and the P extent of the states
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
  using Lds = StateLds<T, MP, NB>;
  constexpr bool kFold = Lds::kFold;  // the intra-chunk parts of dc and dk formed here
  constexpr int oHG = 0;                                         // T [k][t] (Gamma o dY X^T)^T, causal
  constexpr int WSZ = Lds::WSZ;                                  // one chunk's weights and log-decays
  // two chunks' weights (the next one formed during this one's update) when LDS allows
  constexpr int NWB = Lds::NWB;
  constexpr int oW = oHG + 64 * XS * (int)sizeof(T);             // float weights, NWB chunks
  constexpr int oRd = oW + NWB * WSZ * 4;                        // float [8 waves][MPF][Q] token partials
  constexpr int oEx = oRd + 8 * MPF * kQ * 4;                    // float exchange
  constexpr int oSc = oEx + Ex::kFloats * 4;                     // float rates, log tau, scales
  constexpr int oHH = (oSc + 4 * MP * 4 + 15) / 16 * 16;         // T [t][k] H = (C B^T) o (dY X^T), causal
  __shared__ __align__(16) unsigned char sm[oHH + (kFold ? Lds::kHH : 16)];
  T* HGT = reinterpret_cast<T*>(sm + oHG);
  T* HH = reinterpret_cast<T*>(sm + oHH);
  float* const W0 = reinterpret_cast<float*>(sm + oW);
  float* const W1 = W0 + (NWB - 1) * WSZ;
  float* redZ = reinterpret_cast<float*>(sm + oRd);
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
    if constexpr (kFold) HH[i] = (T)0.0f;
    Xb0[i] = Yb0[i] = (T)0.0f;
    Xb1[Cfg::NBUF == 2 ? i : 0] = Yb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;
  }
  for (int i = tid; i < 64 * BS; i += 512) Bb0[i] = Bb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;
  for (int i = tid; i < 64 * CS; i += 512) Cb[i] = (T)0.0f;

  // ---- state S^T: S[m][pb] holds mode mo + m, rows p = 16 pb + 4 lg + r, column ncol
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)p.Mall * N * Ps;
  floatx4 S[MPF][4];
  {
    int lo = ncol * Ps + lg * 4;
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
            v = p.init_state[sbase + (int64_t)(mo + m) * N * Ps + lo + pb * 16 + r];
          S[m][pb][r] = v;
        }
  }

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * Ps;
  const T* yg = reinterpret_cast<const T*>(p.dy) + (((int64_t)b * L) * H + h) * Ps;
  const T* Bgp = reinterpret_cast<const T*>(p.Bm) + (((int64_t)b * L) * G + g) * N;
  const T* Cgp = reinterpret_cast<const T*>(p.Cm) + (((int64_t)b * L) * G + g) * N;
  const int64_t xstride = (int64_t)H * Ps, bstride = (int64_t)G * N;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const int64_t lg_st = (int64_t)H * p.Mall;
  const float* lse_bh = BLK ? p.lse + ((int64_t)b * L * H + h) * 2 : nullptr;  // [t][H][2]
  PairLogits<MP, 512, BLK> lgt_n;  // the logits (and normalizers) of the next chunk's weight pass
  auto load_controls = [&](int c, float& dtv, float& al, float& lam) {
    const int tg = c * kQ + lane;
    const bool valid = tg < L;
    dtv = valid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al = valid ? al_bh[tg * p.as1] : 1.0f;
    lam = (valid && lm_bh) ? lm_bh[tg * p.ls1] : 1.0f;
    lgt_n.load(rl_bh, wl_bh, c * kQ, min(kQ, L - c * kQ), M, lg_st, threadIdx.x, lse_bh, (int64_t)H * 2);
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
  const int64_t bh_i = (int64_t)b * H + h;
  float* dcg = wk.dc + ((int64_t)ps * p.Bsz * H * L + bh_i * L) * p.Mall;  // this head's dc partial [L][Mall]

  // Per-(token, mode) weights of chunk c into Wd, from the controls in dt_n, al_n,
  // lam_n.  Chunk c + 1's weights are formed at the end of chunk c's step, so that
  // their latency overlaps that step's state update.
  int unsafe_c = 0;  // modes past the factorisation bound
  auto weights = [&](int c, float* Wd) __attribute__((always_inline)) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    const ChunkCtl k = chunk_controls(dt_n, al_n, lam_n, lm_bh != nullptr, nv);
    float* lh = Wd + NWA * SW;
    chunk_log_decays<MP, 8>(k.dtt, s_rr, lh, lh + SW);
    barrier();  // log-decays in LDS
    unsafe_c = pair_weights<MP, kState, 512, BLK>(k, nv, M, lgt_n, rl_bh == wl_bh, s_rr, s_lnt, lh, lh + SW,
                                                  s_E2 + (c & 1) * MP, s_E2 + ((c + 1) & 1) * MP, Wd);
  };
  barrier();  // rates and scales in LDS
  if constexpr (NWB == 2) weights(0, W0);

  auto step = [&](int c, T* Xc, T* Yc, T* Bc, T* Xn, T* Yn, T* Bn, float* W, float* Wn)
                  __attribute__((always_inline)) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    // lane-derived addresses recomputed per chunk rather than held across the loop
    const int tid = fresh_tid(), lane = tid & 63, li = lane & 15, lg = lane >> 4;
    const float* Ecur = s_E2 + (c & 1) * MP;
    const float* P_O = W;             // c e^{-l} (c past the factorisation bound)
    const float* P_Vt = W + 1 * SW;   // kappa e^{l} (kappa)
    const float* P_wdc = W + 2 * SW;  // c e^{-l} E: the readout weight of dC
    const float* P_v = W + 3 * SW;
    const float* P_lh = W + NWA * SW;
    const float* P_ll = P_lh + SW;
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
      const float Enew = uniform(Ecur[mo + m] * fexp(-P_lh[(mo + m) * kWQ + kQ - 1]));
      renf[m] = Enew;
      if (__float_as_int(Enew) < __float_as_int(kRescaleFloor)) renbits |= 1 << m;
    }

    __builtin_amdgcn_sched_barrier(0);
    // ---- intra-chunk tiles: HG = Gamma o D (LDS, transposed); the tiles of the reverse sweeps
    {
#pragma unroll
      for (int jt = 0; jt < 2; ++jt) {
        const int tile = wave + 8 * jt;
        if (tile >= kTiles) break;
        const int tb = tile_row(tile), kb = tile_col(tile);
        const floatx4 D = dyx_tile<T, XS>(Yc, Xc, tb, kb, tid);
        floatx4 Gm = rank_m_tile<MP>(P_O, P_Vt, tb * 16, kb * 16, unsafe, tid);
        if (unsafe) unsafe_terms<MP>(Gm, unsafe, P_O, P_Vt, P_lh, P_ll, tb, kb, tid);
        float hv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r, kk = kb * 16 + li;
          hv[r] = keep_if_ge(Gm[r] * D[r], t, kk);
        }
        T* dst = HGT + (kb * 16 + li) * XS + tb * 16 + lg * 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[r] = (T)hv[r];
        if constexpr (kFold) {
          T* hh = HH + (tb * 16 + lg * 4) * XS + kb * 16 + li;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            hh[r * XS] = (T)keep_if_ge(gcur.get(jt, r) * D[r], tb * 16 + lg * 4 + r, kb * 16 + li);
        }
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
      }
    }

    if (c + 1 < nchunks) gtile.load(gtiles + (((int64_t)b * nchunks + c + 1) * G + g) * (kTiles * kTileElems), wave, lane);

    __builtin_amdgcn_sched_barrier(0);
    // ---- readout side of the state entering the chunk, transposed: U^T_m = S_m dY^T
    // (rows n of this wave's block, columns t), dC^T (inter) and per mode
    // z_{t,m} = C_t . (S_m dy_t) over this wave's rows of N
    floatx4 dCa[4];  // dC^T: rows n = 16 nb + 4 lg + r, column t = 16 tb + li
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) dCa[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (active) {
      {
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
          const T* crow = Cb + (tb * 16 + li) * CS + nb * 16 + lg * 4;
          float cv[4];
          load4(crow, cv);
#pragma unroll
          for (int m = 0; m < MPF; ++m) {
            floatx4 U = {0.f, 0.f, 0.f, 0.f};
            mma(U, Sa[m][0], y0);
            mma(U, Sa[m][1], y1);
            const float wd = P_wdc[(mo + m) * kWQ + tb * 16 + li];
#pragma unroll
            for (int r = 0; r < 4; ++r) dCa[tb][r] += wd * U[r];
            // z over this lane's 4 rows of N, then over the 4 lane groups (16 rows)
            const float z = xor32_sum(xor16_sum(U[0] * cv[0] + U[1] * cv[1] + U[2] * cv[2] + U[3] * cv[3]));
            if (lg == 0) redZ[(wave * MPF + m) * kQ + tb * 16 + li] = z;
          }
        }
        if (Cfg::NACT > 1) Ex::put(XCH, wave, part, dCa);
      }
    }
    barrier();  // HG, token partials and exchange complete; C is free
    if (Cfg::NBUF == 2 && c + 1 < nchunks) stageC(c + 1);

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

    __builtin_amdgcn_sched_barrier(0);
    // ---- the state part of dL/dc over this workgroup's rows of N: e^{-l_t} E_m times
    // the sum over the N blocks (in order) of z; with the intra-chunk products here,
    // the first workgroup of the head adds sum_{k<=t} H_{t,k} kappa_{k,m} e^{-(l_t - l_k)}
    // (waves 0..3, row block = wave) and the last forms the intra-chunk part of dk,
    // sum_{t'>=t} H_{t',t} c_{t',m} e^{-(l_t' - l_t)} (waves 4..7, column block = wave - 4)
    if constexpr (!kFold) {
      for (int i = tid; i < kQ * MP; i += 512) {
        const int t = i / MP, m = i - t * MP;
        if (m < M && t < nv) {
          const int pt = m / MPF, j = m - pt * MPF;
          float z = 0.0f;
#pragma unroll
          for (int q = 0; q < NBF; ++q) z += redZ[((pt * NBF + q) * MPF + j) * kQ + t];
          dcg[(int64_t)(t0 + t) * p.Mall + m] = fexp(-P_lh[m * kWQ + t]) * Ecur[m] * z;
        }
      }
    } else {
      const int tb = wave & 3;
      const bool cside = wave < 4;
      const bool intra = cside ? ps == 0 : ps == Cfg::PS - 1;
      constexpr int MB = (MP + 15) / 16;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int m = mb * 16 + li;
        const int mm = m < MP ? m : 0;
        const bool fac = m < MP && !((unsafe >> mm) & 1);
        const bool direct = m < M && ((unsafe >> mm) & 1);
        const float* lhm = P_lh + mm * kWQ;
        const float* llm = P_ll + mm * kWQ;
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
        if (intra) {
          if (cside) {
            for (int kq = 0; kq < (tb + 1) * 4; ++kq) {
              const int kk = kq * 4 + lg;
              acc = __builtin_amdgcn_mfma_f32_16x16x4f32(to_f32(HH[(tb * 16 + li) * XS + kk]),
                                                         fac ? P_Vt[mm * kWQ + kk] : 0.0f, acc, 0, 0, 0);
            }
          } else {
            for (int tq = tb * 4; tq < 16; ++tq) {
              const int t = tq * 4 + lg;
              acc = __builtin_amdgcn_mfma_f32_16x16x4f32(to_f32(HH[t * XS + tb * 16 + li]),
                                                         fac ? P_O[mm * kWQ + t] : 0.0f, acc, 0, 0, 0);
            }
          }
        }
        // modes past the factorisation bound: one exponential per pair, the lane's four
        // rows in one loop
        float dsum[4] = {0.f, 0.f, 0.f, 0.f};
        if (intra && direct) {
          const int tr0 = tb * 16 + lg * 4;
          if (cside) {
            for (int kk = 0; kk <= tr0 + 3; ++kk) {
              const float v = P_Vt[mm * kWQ + kk];
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (kk <= tr0 + r) dsum[r] += to_f32(HH[(tr0 + r) * XS + kk]) * v * ell_decay(lhm, llm, tr0 + r, kk);
            }
          } else {
            for (int t2 = tr0; t2 < 64; ++t2) {
              const float v = P_O[mm * kWQ + t2];
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (t2 >= tr0 + r) dsum[r] += to_f32(HH[t2 * XS + tr0 + r]) * v * ell_decay(lhm, llm, t2, tr0 + r);
            }
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r;
          if (cside) {
            float z = 0.0f;
            if (m < M) {
              const int pt = m / MPF, j = m - pt * MPF;
#pragma unroll
              for (int q = 0; q < NBF; ++q) z += redZ[((pt * NBF + q) * MPF + j) * kQ + t];
            }
            float v = (m < M ? Ecur[mm] : 0.0f) * z;
            if (intra && !direct) v += acc[r];
            const float dc = fexp(-lhm[t]) * v + dsum[r];
            if (m < M && t < nv) dcg[(int64_t)(t0 + t) * p.Mall + m] = dc;
          } else if (intra) {
            const float dk = direct ? dsum[r] : fexp(lhm[t]) * acc[r];
            if (m < M && t < nv) wk.dki[(bh_i * L + t0 + t) * p.Mall + m] = dk;
          }
        }
      }
    }
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

  // ---- final-state term <dS_final_m, S_final_m> per mode over this workgroup's rows of N,
  // and sum(dy . x); per wave over its lanes, then over the waves in order
  float fpart[MPF];
#pragma unroll
  for (int m = 0; m < MPF; ++m) fpart[m] = 0.0f;
  if (p.d_final_state && active) {
    const float* Ef = s_E2 + (nchunks & 1) * MP;
    int lo = ncol * Ps + lg * 4;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MPF; ++m) {
      const float scale = (mo + m < M) ? Ef[mo + m] : 0.0f;
#pragma unroll
      for (int pb = 0; pb < 4; ++pb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pr = pb * 16 + lg * 4 + r;
          if (mo + m < M && ncol < N && pr < P)
            fpart[m] += scale * S[m][pb][r] * p.d_final_state[sbase + (int64_t)(mo + m) * N * Ps + lo + pb * 16 + r];
        }
    }
  }
  float* red = redZ;  // the token partials are no longer needed
#pragma unroll
  for (int m = 0; m < MPF; ++m) {
    const float v = group_allreduce<64>(fpart[m], [](float x, float y) { return x + y; });
    if (lane == 0) red[wave * MPF + m] = v;
  }
  {
    const float v = group_allreduce<64>(dd_acc, [](float x, float y) { return x + y; });
    if (lane == 0) red[8 * MPF + wave] = v;
  }
  barrier();
  if (tid < M) {  // mode tid: the waves holding it, N blocks in order
    const int pt = tid / MPF, j = tid - pt * MPF;
    float fs = 0.f;
    for (int q = 0; q < NBF; ++q) fs += red[(pt * NBF + q) * MPF + j];
    wk.F[((int64_t)ps * p.Bsz * H + bh_i) * p.Mall + tid] = fs;
  }
  if (tid == 0 && ps == 0) {
    float ds = 0.f;
    for (int w2 = 0; w2 < 8; ++w2) ds += red[8 * MPF + w2];
    wk.dDp[bh_i] = ds;
  }
}

// ------------------------------------------------------------- cols sweep

template <typename T, int MP, int NB, bool BLK = false>
__global__ void __launch_bounds__(512) frac_bwd_cols_kernel(ScanParams p, BwdWork wk) {
  using Cfg = ColCfg<T, MP, NB>;
  constexpr int NP = Cfg::NP, XS = Cfg::XS, CS = Cfg::BS;  // C is read transposed here
  constexpr int NBF = Cfg::NBF, FPART = Cfg::FPART, MPF = Cfg::MPF;
  using Ex = Exchange<Cfg::NACT>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M, G = p.G;
  const int Ps = p.Pst;  // row stride of x, dy, dx and the P extent of the states
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
  constexpr int oEx = oW + (NWA + 2) * MP * kWQ * 4;
  constexpr int oSc = oEx + Ex::kFloats * 4;
  __shared__ __align__(16) unsigned char sm[oSc + 4 * MP * 4];
  T* HG = reinterpret_cast<T*>(sm + oHG);
  float* W = reinterpret_cast<float*>(sm + oW);
  float* P_lh = W + NWA * MP * kWQ;  // chunk log-decays, hi and lo parts
  float* P_ll = P_lh + MP * kWQ;
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
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)p.Mall * N * Ps;
  floatx4 Gs[MPF][4];
  {
    int lo = ncol * Ps + lg * 4;
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
            v = p.d_final_state[sbase + (int64_t)(mo + m) * N * Ps + lo + pb * 16 + r];
          Gs[m][pb][r] = v;
        }
  }

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * Ps;
  const T* yg = reinterpret_cast<const T*>(p.dy) + (((int64_t)b * L) * H + h) * Ps;
  const T* Cgp = reinterpret_cast<const T*>(p.Cm) + (((int64_t)b * L) * G + g) * N;
  const int64_t xstride = (int64_t)H * Ps, bstride = (int64_t)G * N;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const int64_t lg_st = (int64_t)H * p.Mall;
  const float* lse_bh = BLK ? p.lse + ((int64_t)b * L * H + h) * 2 : nullptr;  // [t][H][2]
  PairLogits<MP, 512, BLK> lgt_n;  // the logits (and normalizers) of the next chunk's weight pass
  auto load_controls = [&](int c, float& dtv, float& al, float& lam) {
    const int tg = c * kQ + lane;
    const bool valid = tg < L;
    dtv = valid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al = valid ? al_bh[tg * p.as1] : 1.0f;
    lam = (valid && lm_bh) ? lm_bh[tg * p.ls1] : 1.0f;
    lgt_n.load(rl_bh, wl_bh, c * kQ, min(kQ, L - c * kQ), M, lg_st, threadIdx.x, lse_bh, (int64_t)H * 2);
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
    const PairLogits<MP, 512, BLK> lgt = lgt_n.pinned_copy();
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
    chunk_log_decays<MP, 8>(k.dtt, s_rr, P_lh, P_ll);
    barrier();  // log-decays in LDS
    const int unsafe = pair_weights<MP, kCols, 512, BLK>(k, nv, M, lgt, rl_bh == wl_bh, s_rr, s_lnt, P_lh, P_ll, Ecur,
                                                         Enext, W);
    float renf[MPF];
    int renbits = 0;
#pragma unroll
    for (int m = 0; m < MPF; ++m) {
      const float Enew = uniform(Ecur[mo + m] * fexp(-P_lh[(mo + m) * kWQ + kQ - 1]));
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

template <typename T, int MP, int NB, bool BLK = false>
__global__ void __launch_bounds__(512) frac_bwd_rows_kernel(ScanParams p, BwdWork wk) {
  using Cfg = RowCfg<T, MP, NB>;
  constexpr int NP = Cfg::NP, XS = Cfg::XS, BS = Cfg::BS, CS = Cfg::CS;
  constexpr int NPART = Cfg::NPART, MPW = Cfg::MPW, NBW = Cfg::NBW, KBW = Cfg::KBW, TBP = Cfg::TBP;
  using Ex = Exchange<NPART>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M, G = p.G;
  const int Ps = p.Pst;  // row stride of x, dy, dx and the P extent of the states
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
  constexpr int oRd = oW + (NWA + 2) * MP * kWQ * 4;             // float [8 waves][MPW][Q] token partials
  constexpr int oEx = oRd + 8 * MPW * kQ * 4;
  constexpr int oSc = oEx + Ex::kFloats * 4;
  __shared__ __align__(16) unsigned char sm[oSc + 4 * MP * 4];
  T* GG = reinterpret_cast<T*>(sm + oGG);
  T* Dxb = reinterpret_cast<T*>(sm + oDx);
  float* W = reinterpret_cast<float*>(sm + oW);
  float* P_lh = W + NWA * MP * kWQ;  // chunk log-decays, hi and lo parts
  float* P_ll = P_lh + MP * kWQ;
  float* redW = reinterpret_cast<float*>(sm + oRd);
  float* XCH = reinterpret_cast<float*>(sm + oEx);
  float* s_rr = reinterpret_cast<float*>(sm + oSc);
  float* s_lnt = s_rr + MP;
  float* s_E2 = s_lnt + MP;
  constexpr int SW = MP * kWQ;  // stride of the weight arrays
  const float* P_wdx = W;          // kappa e^{-(l_Q-l)} E: the adjoint weight of dx
  const float* P_dE = W + 1 * SW;   // e^{-(l_Q-l)} E: the adjoint weight of dL/dkappa
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
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)p.Mall * N * Ps;
  floatx4 Gs[MPW][NBW];
  {
    int lo = (mo * N + nbo * 16 + lg * 4) * Ps + pc;
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
            v = p.d_final_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * Ps];
          Gs[m][jb][r] = v;
        }
  }
  const float Dh = p.D ? p.D[h] : 0.0f;

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * Ps;
  const T* yg = reinterpret_cast<const T*>(p.dy) + (((int64_t)b * L) * H + h) * Ps;
  T* dxg = reinterpret_cast<T*>(p.dx) + (((int64_t)b * L) * H + h) * Ps;
  const T* Bgp = reinterpret_cast<const T*>(p.Bm) + (((int64_t)b * L) * G + g) * N;
  const T* Cgp = reinterpret_cast<const T*>(p.Cm) + (((int64_t)b * L) * G + g) * N;
  const int64_t xstride = (int64_t)H * Ps, bstride = (int64_t)G * N;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const int64_t lg_st = (int64_t)H * p.Mall;
  const float* lse_bh = BLK ? p.lse + ((int64_t)b * L * H + h) * 2 : nullptr;  // [t][H][2]
  PairLogits<MP, 512, BLK> lgt_n;  // the logits (and normalizers) of the next chunk's weight pass
  auto load_controls = [&](int c, float& dtv, float& al, float& lam) {
    const int tg = c * kQ + lane;
    const bool valid = tg < L;
    dtv = valid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al = valid ? al_bh[tg * p.as1] : 1.0f;
    lam = (valid && lm_bh) ? lm_bh[tg * p.ls1] : 1.0f;
    lgt_n.load(rl_bh, wl_bh, c * kQ, min(kQ, L - c * kQ), M, lg_st, threadIdx.x, lse_bh, (int64_t)H * 2);
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
  float* dkg = wk.dk + ((int64_t)ps * p.Bsz * H * L + ((int64_t)b * H + h) * L) * p.Mall;  // [L][Mall]
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
    const PairLogits<MP, 512, BLK> lgt = lgt_n.pinned_copy();
    const TilePrefetch<T> gcur = ggt.pinned_copy();
    if (Cfg::kBf16 && i > 0 && !(BLK && p.y_part)) store_dx(c + 1);
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
    chunk_log_decays<MP, 8>(k.dtt, s_rr, P_lh, P_ll);
    barrier();  // log-decays in LDS
    const int unsafe = pair_weights<MP, kRows, 512, BLK>(k, nv, M, lgt, rl_bh == wl_bh, s_rr, s_lnt, P_lh, P_ll, Ecur,
                                                         Enext, W);
    float renf[MPW];
    int renbits = 0;
#pragma unroll
    for (int m = 0; m < MPW; ++m) {
      const float Enew = uniform(Ecur[mo + m] * fexp(-P_lh[(mo + m) * kWQ + kQ - 1]));
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
    // and per mode w_{t,m} = (B_t^T G_m) . x_t over this wave's columns (and rows) of the adjoint
    floatx4 dxa[4];  // dx^T: rows p = 16 pb + 4 lg + r, column t = 16 tb + li
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) dxa[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    {
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
#pragma unroll
            for (int q = 0; q < TBP; ++q) {
              const int tb = tp * TBP + q;
              floatx4 Z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
              for (int kb = 0; kb < KBW; ++kb) mma(Z, Gf[kb], Ba[q][kb]);
              const float wx = P_wdx[(mo + m) * kWQ + tb * 16 + li];
#pragma unroll
              for (int r = 0; r < 4; ++r) dxa[tb][r] = __builtin_fmaf(wx, Z[r], dxa[tb][r]);
              // w over this lane's 4 columns of P, then over the 4 lane groups (16 columns)
              float xv[4];
              load4(Xb + (tb * 16 + li) * XS + pb * 16 + lg * 4, xv);
              const float wv = xor32_sum(xor16_sum(Z[0] * xv[0] + Z[1] * xv[1] + Z[2] * xv[2] + Z[3] * xv[3]));
              if (lg == 0) redW[(wave * MPW + m) * kQ + tb * 16 + li] = wv;
            }
          }
        }
        if (NPART > 1) Ex::put(XCH, wave, part, dxa);
      } else {
        // waves without adjoint columns add nothing
        for (int i2 = lane; i2 < MPW * kQ; i2 += 64) redW[wave * MPW * kQ + i2] = 0.0f;
      }
    }
    barrier();  // GG, exchange and token partials complete; B and x are free
    if (Cfg::NBUF == 2 && c > 0) stage_early(c - 1);

    // ---- the adjoint part of dL/dkappa over this workgroup's columns of P:
    // e^{-(l_Q - l_t)} E_m times the sum over the waves holding mode m (in order) of w
    for (int i2 = tid; i2 < kQ * MP; i2 += 512) {
      const int t = i2 / MP, m = i2 - t * MP;
      if (m < M && t < nv) {
        float wsum = 0.0f;
#pragma unroll
        for (int w2 = 0; w2 < 8; ++w2) {
          const int q = w2 / Cfg::NPW, mo2 = Cfg::kModeSplit ? q * MPW : 0;
          if (q < NPART && m >= mo2 && m < mo2 + MPW) wsum += redW[(w2 * MPW + (m - mo2)) * kQ + t];
        }
        dkg[(int64_t)(t0 + t) * p.Mall + m] = P_dE[m * kWQ + t] * wsum;
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
      floatx4 v = dxa[tb];
      if constexpr (BLK) {  // a mode block: float32 partial sums across the blocks
        // a wave-uniform 64-bit base and a 32-bit lane offset: a per-lane 64-bit index
        // spilled here and its reload waited on every outstanding copy
        const int64_t xi = (((int64_t)b * L + t0) * H + h) * Ps + (int64_t)(t * H * Ps + pr);
        if (t < nv && pr < P) {
          if (p.y_in) {
            const float4 u = *reinterpret_cast<const float4*>(p.y_in + xi);
            v[0] += u.x;
            v[1] += u.y;
            v[2] += u.z;
            v[3] += u.w;
          }
          if (p.y_part) *reinterpret_cast<float4*>(p.y_part + xi) = make_float4(v[0], v[1], v[2], v[3]);
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] += Dh * yv[r];
      if (!(BLK && p.y_part)) {
        if (Cfg::kBf16) store4(Dxb + t * XS + pr, v);  // staged, stored 16 bytes at a time
        else if (t < nv && pr < P) store4(dxg + (int64_t)t0 * xstride + t * xstride + pr, v);
      }
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
  if (Cfg::kBf16 && !(BLK && p.y_part)) store_dx(0);

  // ---- the adjoint of the state before token 0 (this workgroup's columns of P)
  if (p.dinit_state && active) {
    const float* Ef = s_E2 + (nchunks & 1) * MP;
    // lane offset kept opaque (as for the initial load) so that no per-element offset
    // of this store is formed before, and held across, the sequence loop
    int lo = (mo * N + nbo * 16 + lg * 4) * Ps + pc;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MPW; ++m)
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = (nbo + jb) * 16 + lg * 4 + r;
          if (mo + m < M && n < N && pc < P)
            p.dinit_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * Ps] = Gs[m][jb][r] * Ef[mo + m];
        }
  }

  // ---- the initial-state term <S_init, dS_init> per mode over this workgroup's columns:
  // per wave, then over the waves holding each mode in a fixed order
  barrier();  // the token partials are no longer read
  {
    const float* Ef = s_E2 + (nchunks & 1) * MP;
    int lo = (mo * N + nbo * 16 + lg * 4) * Ps + pc;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MPW; ++m) {
      float ip = 0.0f;
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = (nbo + jb) * 16 + lg * 4 + r;
          if (p.init_state && active && mo + m < M && n < N && pc < P)
            ip += p.init_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * Ps] * Gs[m][jb][r];
        }
      ip = group_allreduce<64>(ip, [](float x, float y) { return x + y; });
      if (lane == 0) redW[wave * MPW + m] = (active && mo + m < M) ? ip * Ef[mo + m] : 0.0f;
    }
  }
  barrier();
  if (tid < M) {
    float s = 0.0f;
    for (int w = 0; w < 8; ++w) {
      const int pw = w / Cfg::NPW;
      const int mow = Cfg::kModeSplit ? pw * MPW : 0;
      if (pw < NPART && tid >= mow && tid < mow + MPW) s += redW[w * MPW + tid - mow];
    }
    wk.I[((int64_t)ps * p.Bsz * H + (int64_t)b * H + h) * p.Mall + tid] = s;
  }
}

// ------------------------------------------------------ intra-chunk parts
//
// The intra-chunk parts of dL/dc and dL/dkappa, one workgroup of four waves per
// (batch, chunk, head), independent of every other chunk:
//   dc_{t,m} += sum_{k<=t} H_{t,k} kappa_{k,m} e^{-(l_t - l_k)}
//   dk_{k,m} += sum_{t>=k} H_{t,k} c_{t,m} e^{-(l_t - l_k)}
//   H = (C B^T) o (dY X^T)   (causal)
// as float32 matrix-core products e^{-l_t} (H kappa e^{l})_t and e^{l_k} (H^T c e^{-l})_k
// for the modes whose chunk decay stays below the factorisation bound, one
// exponential per pair for the others.
template <typename T, int MP, bool BLK = false>
__global__ void __launch_bounds__(256) frac_bwd_intra_kernel(ScanParams p, const T* __restrict__ gtiles,
                                                             float* __restrict__ dc_out, float* __restrict__ dk_out) {
  constexpr bool kBf16 = sizeof(T) == 2;
  constexpr int XS = kBf16 ? 64 + 8 : 64 + 4;
  constexpr int HS = kWQ;  // float H [t][k]
  constexpr int MB = (MP + 15) / 16;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, M = p.M, G = p.G;
  const int Ps = p.Pst;
  const int nchunks = (L + kQ - 1) / kQ;
  // block = (b, c, h), heads fastest: the heads of a group read the same C B^T tiles
  const int h = (int)(blockIdx.x % H);
  const int bc = (int)(blockIdx.x / H);
  const int c = bc % nchunks, b = bc / nchunks;
  const int g = h * G / H;
  const int t0 = c * kQ, nv = min(kQ, L - t0);

  __shared__ __align__(16) T Xs[64 * XS], Ys[64 * XS];
  __shared__ __align__(16) float Hs[64 * HS];
  __shared__ __align__(16) float W[4 * MP * kWQ];
  __shared__ float s_rr[MP], s_lnt[MP];
  float* P_O = W;                 // c e^{-l} (c past the factorisation bound)
  float* P_Vt = W + MP * kWQ;     // kappa e^{l} (kappa)
  float* P_lh = W + 2 * MP * kWQ; // chunk log-decays, hi and lo parts
  float* P_ll = W + 3 * MP * kWQ;

  if (tid < MP) {
    const float tau = (tid < M) ? p.tau[tid] : 1.0f;
    s_rr[tid] = (tid < M) ? 1.0f / tau : 0.0f;
    s_lnt[tid] = (tid < M) ? logf(tau) : 0.0f;
  }
  for (int i = tid; i < 64 * HS; i += 256) Hs[i] = 0.0f;
  // x and dy of the chunk, 16 bytes per thread (columns past P, tokens past the sequence: zero)
  {
    constexpr int E16 = 16 / (int)sizeof(T), CPR = 64 / E16;
    const int64_t xstride = (int64_t)H * Ps;
    const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L + t0) * H + h) * Ps;
    const T* yg = reinterpret_cast<const T*>(p.dy) + (((int64_t)b * L + t0) * H + h) * Ps;
    for (int i = tid; i < 64 * CPR; i += 256) {
      const int t = i / CPR, col = (i - t * CPR) * E16;
      int4 vx = make_int4(0, 0, 0, 0), vy = vx;
      if (t < nv && col < P) {
        vx = *reinterpret_cast<const int4*>(xg + t * xstride + col);
        vy = *reinterpret_cast<const int4*>(yg + t * xstride + col);
      }
      *reinterpret_cast<int4*>(Xs + t * XS + col) = vx;
      *reinterpret_cast<int4*>(Ys + t * XS + col) = vy;
    }
  }
  // per-token controls (lane = token, every wave) and the (token, mode) logits
  const bool tv = lane < nv;
  const int64_t tok = ((int64_t)b * L + t0 + lane) * H + h;
  const float dtv = tv ? p.dt[tok] : 0.0f;
  const float al = tv ? strided3(p.alpha, p.as0, p.as1, p.as2, b, t0 + lane, h) : 1.0f;
  const float lam = (tv && p.lambda) ? strided3(p.lambda, p.ls0, p.ls1, p.ls2, b, t0 + lane, h) : 1.0f;
  const ChunkCtl k = chunk_controls(dtv, al, lam, p.lambda != nullptr, nv);
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  PairLogits<MP, 256, BLK> lgt;
  lgt.load(rl_bh, wl_bh, t0, nv, M, (int64_t)H * p.Mall, tid, BLK ? p.lse + ((int64_t)b * L * H + h) * 2 : nullptr,
           (int64_t)H * 2);
  __syncthreads();  // rates, zeroed H, x and dy in LDS
  chunk_log_decays<MP, 4>(k.dtt, s_rr, P_lh, P_ll);
  __syncthreads();  // log-decays in LDS
  const int unsafe = pair_weights<MP, kIntra, 256, BLK>(k, nv, M, lgt, rl_bh == wl_bh, s_rr, s_lnt, P_lh, P_ll,
                                                        nullptr, nullptr, W);
  // ---- H = (C B^T) o (dY X^T), causal tiles [t][k]
  const T* gt = gtiles + (((int64_t)b * nchunks + c) * G + g) * (kTiles * kTileElems);
  for (int tile = wave; tile < kTiles; tile += 4) {
    const int tb = tile_row(tile), kb = tile_col(tile);
    const floatx4 D = dyx_tile<T, XS>(Ys, Xs, tb, kb, tid);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = tb * 16 + lg * 4 + r, kk = kb * 16 + li;
      Hs[t * HS + kk] = keep_if_ge(to_f32(gt[tile * kTileElems + lane * 4 + r]) * D[r], t, kk);
    }
  }
  __syncthreads();  // H and the weights in LDS

  // ---- tokens of row block tb = wave (dc) and column block tb (dk), modes as columns
  const int tb = wave;
  const int64_t obase = (((int64_t)b * H + h) * L + t0) * p.Mall;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = mb * 16 + li;
    const int mm = m < MP ? m : 0;
    const bool fac = m < MP && !((unsafe >> mm) & 1);
    floatx4 cI = {0.f, 0.f, 0.f, 0.f}, kI = {0.f, 0.f, 0.f, 0.f};
    for (int kq = 0; kq < (tb + 1) * 4; ++kq) {
      const int kk = kq * 4 + lg;
      cI = __builtin_amdgcn_mfma_f32_16x16x4f32(Hs[(tb * 16 + li) * HS + kk], fac ? P_Vt[mm * kWQ + kk] : 0.0f, cI,
                                                0, 0, 0);
    }
    for (int tq = tb * 4; tq < 16; ++tq) {
      const int t = tq * 4 + lg;
      kI = __builtin_amdgcn_mfma_f32_16x16x4f32(Hs[t * HS + tb * 16 + li], fac ? P_O[mm * kWQ + t] : 0.0f, kI, 0, 0,
                                                0);
    }
    const bool direct = m < M && ((unsafe >> mm) & 1);
    const float* lhm = P_lh + mm * kWQ;
    const float* llm = P_ll + mm * kWQ;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = tb * 16 + lg * 4 + r;
      float dc, dk;
      if (!direct) {
        dc = fexp(-lhm[t]) * cI[r];
        dk = fexp(lhm[t]) * kI[r];
      } else {
        dc = dk = 0.0f;
        for (int kk = 0; kk <= t; ++kk) dc += Hs[t * HS + kk] * P_Vt[mm * kWQ + kk] * ell_decay(lhm, llm, t, kk);
        for (int t2 = t; t2 < 64; ++t2) dk += Hs[t2 * HS + t] * P_O[mm * kWQ + t2] * ell_decay(lhm, llm, t2, t);
      }
      if (m < M && t < nv) {
        dc_out[obase + (int64_t)t * p.Mall + m] = dc;
        dk_out[obase + (int64_t)t * p.Mall + m] = dk;
      }
    }
  }
}

// dB, dC of each group: fixed-order sum of the per-head partials (over the mode
// blocks, then the group's heads); each thread sums 16 bytes of a (token, group) row.
template <typename T>
__global__ void __launch_bounds__(256) frac_bwd_group_sum_kernel(ScanParams p, const T* __restrict__ dBp,
                                                                 const T* __restrict__ dCp, int64_t nrows, int nslot,
                                                                 int64_t slot_stride) {
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
  for (int q = 0; q < nslot; ++q)
    for (int j = 0; j < hpg; ++j) {
      const int64_t off = q * slot_stride + (bt * H + g * hpg + j) * N + ch * E;
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

constexpr int kModeBlock = 8;  // modes per launch of the mode-block backward

// Workgroups per head of the state sweep (along N) and of the rows sweep (along P),
// as ColCfg and RowCfg choose them.
int pad_modes(int M) { return M <= 1 ? 1 : M <= 2 ? 2 : M <= 4 ? 4 : 8; }
int state_parts(const ScanParams& p) { return pad_modes(p.M) * (p.NP / 16) > 32 ? 2 : 1; }
int rows_parts(const ScanParams& p) { return (pad_modes(p.M) >= 8 && p.io_bf16) ? 2 : 1; }
int mode_blocks(const ScanParams& p) { return p.Mall > kModeBlock ? (p.Mall + kModeBlock - 1) / kModeBlock : 1; }
int column_groups(const ScanParams& p) { return (p.Pst + 63) / 64; }

// Workspace: C B^T tiles, the state sweep's Gamma tiles, per-head dB / dC partials
// (per mode block and column group), the (token, mode) partials (per sweep part and
// column group), per-mode terms, dD partials, the finisher's tile sums; with mode
// blocks also the log-normalizers and the float32 partial dx.
struct BwdLayout {
  size_t tiles, gg, hg, dBp, dCp, dc, dk, dki, F, I, dDp, gtl, lse, dxp, total;
};

BwdLayout bwd_layout(const ScanParams& p) {
  BwdLayout l{};
  const size_t es = p.io_bf16 ? 2 : 4;
  const size_t bl = (size_t)p.Bsz * p.L, blhm = bl * p.H * p.Mall, bh = (size_t)p.Bsz * p.H;
  const size_t nmb = (size_t)mode_blocks(p), R = (size_t)column_groups(p);
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  l.tiles = 0;
  const size_t gtb = (size_t)p.Bsz * ((p.L + kQ - 1) / kQ) * p.H * kTiles * kTileElems * es;
  l.gg = up(cb_tiles_bytes(p));
  l.hg = l.gg + up(gtb);
  l.dBp = l.hg + up(gtb);
  l.dCp = l.dBp + up(R * nmb * bl * p.H * p.N * es);
  l.dc = l.dCp + up(R * nmb * bl * p.H * p.N * es);
  l.dk = l.dc + up(sizeof(float) * R * (state_parts(p) + 1) * blhm);
  l.dki = l.dk + up(sizeof(float) * R * rows_parts(p) * blhm);
  l.F = l.dki + up(sizeof(float) * R * blhm);
  l.I = l.F + up(sizeof(float) * R * state_parts(p) * bh * p.Mall);
  l.dDp = l.I + up(sizeof(float) * R * rows_parts(p) * bh * p.Mall);
  l.gtl = l.dDp + up(sizeof(float) * R * bh);
  l.lse = l.gtl + up(grad_tiles_bytes(p));
  l.dxp = l.lse + (nmb > 1 ? up(sizeof(float) * 2 * bl * p.H) : 0);
  l.total = l.dxp + (nmb > 1 ? up(sizeof(float) * bl * p.H * p.Pst) : 0);
  return l;
}

// The three sweeps (and the intra-chunk kernel when the state sweep does not fold
// it in) for the modes and columns p covers.
template <typename T, int MP, int NB, bool BLK>
hipError_t launch_bwd_sweeps(const ScanParams& p, const BwdWork& wk, const T* tiles, size_t blhm, hipStream_t stream) {
  using SC = ColCfg<T, MP, NB>;
  using RC = RowCfg<T, MP, NB>;
  constexpr bool kFold = StateLds<T, MP, NB>::kFold;
  const int bh = p.Bsz * p.H;
  hipLaunchKernelGGL((frac_bwd_state_kernel<T, MP, NB, BLK>), dim3(bh * SC::PS), dim3(512), 0, stream, p, wk);
  hipError_t e;
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((frac_bwd_rows_kernel<T, MP, NB, BLK>), dim3(bh * RC::PS), dim3(512), 0, stream, p, wk);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((frac_bwd_cols_kernel<T, MP, NB, BLK>), dim3(bh * SC::PS), dim3(512), 0, stream, p, wk);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if constexpr (!kFold) {
    const int64_t nblk = (int64_t)p.Bsz * ((p.L + kQ - 1) / kQ) * p.H;
    hipLaunchKernelGGL((frac_bwd_intra_kernel<T, MP, BLK>), dim3((unsigned)nblk), dim3(256), 0, stream, p, tiles,
                       wk.dc + SC::PS * blhm, wk.dki);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename T, int MP, int NB>
hipError_t launch_bwd_variant(const ScanParams& p, void* ws, hipStream_t stream) {
  using SC = ColCfg<T, MP, NB>;
  using RC = RowCfg<T, MP, NB>;
  if (SC::PS != state_parts(p) || RC::PS != rows_parts(p)) return hipErrorInvalidValue;
  const BwdLayout l = bwd_layout(p);
  unsigned char* base = reinterpret_cast<unsigned char*>(ws);
  const size_t blhm = (size_t)p.Bsz * p.L * p.H * p.Mall, bhm = (size_t)p.Bsz * p.H * p.Mall;
  constexpr bool kFold = StateLds<T, MP, NB>::kFold;
  constexpr int NDC = SC::PS + (kFold ? 0 : 1);  // dc slots per column group
  BwdWork wk;
  wk.tiles = base + l.tiles;
  wk.gg = base + l.gg;
  wk.hg = base + l.hg;
  wk.dBp = base + l.dBp;
  wk.dCp = base + l.dCp;
  wk.dc = reinterpret_cast<float*>(base + l.dc);
  wk.dk = reinterpret_cast<float*>(base + l.dk);
  wk.dki = reinterpret_cast<float*>(base + l.dki);
  wk.F = reinterpret_cast<float*>(base + l.F);
  wk.I = reinterpret_cast<float*>(base + l.I);
  wk.dDp = reinterpret_cast<float*>(base + l.dDp);
  hipError_t e = launch_cb_tiles(p, base + l.tiles, stream);
  if (e != hipSuccess) return e;
  const T* tiles = reinterpret_cast<const T*>(base + l.tiles);
  const int nmb = mode_blocks(p), R = column_groups(p);
  float* lse = reinterpret_cast<float*>(base + l.lse);
  if (nmb > 1 && (e = launch_mode_lse(p, lse, stream)) != hipSuccess) return e;
  const size_t slot = (size_t)p.Bsz * p.L * p.H * p.N * sizeof(T);  // one dB / dC partial
  // Per column group of 64 columns of P (independent but for their sums over P, which
  // get their own slots), per block of eight modes: the weights normalised over the
  // bank, dx summed in float32 in block order (the last block adds the skip term).
  for (int r = 0; r < R; ++r) {
    const ScanParams pc = column_group(p, r * 64);
    for (int q = 0; q < nmb; ++q) {
      const int mo = q * kModeBlock;
      ScanParams pb = pc;
      BwdWork wb = wk;
      wb.dBp = reinterpret_cast<unsigned char*>(wk.dBp) + (size_t)(r * nmb + q) * slot;
      wb.dCp = reinterpret_cast<unsigned char*>(wk.dCp) + (size_t)(r * nmb + q) * slot;
      wb.dc = wk.dc + (size_t)r * NDC * blhm + mo;
      wb.dk = wk.dk + (size_t)r * RC::PS * blhm + mo;
      wb.dki = wk.dki + (size_t)r * blhm + mo;
      wb.F = wk.F + (size_t)r * SC::PS * bhm + mo;
      wb.I = wk.I + (size_t)r * RC::PS * bhm + mo;
      wb.dDp = wk.dDp + (size_t)r * p.Bsz * p.H;
      if (nmb == 1) {
        if ((e = launch_bwd_sweeps<T, MP, NB, false>(pb, wb, tiles, blhm, stream)) != hipSuccess) return e;
        continue;
      }
      if constexpr (MP == kModeBlock) {
        const int64_t NPs = (int64_t)p.N * p.Pst;
        float* dxp = reinterpret_cast<float*>(base + l.dxp) + r * 64;
        pb.M = min(kModeBlock, p.Mall - mo);
        pb.tau = p.tau + mo;
        if (p.read_logit) pb.read_logit = p.read_logit + mo;
        if (p.write_logit) pb.write_logit = p.write_logit + mo;
        if (pc.init_state) pb.init_state = pc.init_state + mo * NPs;
        if (pc.d_final_state) pb.d_final_state = pc.d_final_state + mo * NPs;
        if (pc.dinit_state) pb.dinit_state = pc.dinit_state + mo * NPs;
        pb.lse = lse;
        pb.y_in = q > 0 ? dxp : nullptr;
        pb.y_part = q + 1 < nmb ? dxp : nullptr;
        if ((e = launch_bwd_sweeps<T, MP, NB, true>(pb, wb, tiles, blhm, stream)) != hipSuccess) return e;
      } else {
        return hipErrorInvalidValue;
      }
    }
  }
  GradInputs gi;
  gi.dc = wk.dc;
  gi.dk = wk.dk;
  gi.dki = wk.dki;
  gi.ndc = R * NDC;
  gi.ndk = R * RC::PS;
  gi.ndki = R;
  gi.F = wk.F;
  gi.nF = R * SC::PS;
  gi.I = wk.I;
  gi.nI = R * RC::PS;
  gi.dDp = wk.dDp;
  gi.nD = R;
  grad_tiles_at(p, base + l.gtl, gi);
  if ((e = launch_grad_finish(p, gi, stream)) != hipSuccess) return e;
  const int64_t nrows = (int64_t)p.Bsz * p.L;
  const int64_t nthr = nrows * p.G * (p.N / (16 / (int)sizeof(T)));
  hipLaunchKernelGGL((frac_bwd_group_sum_kernel<T>), dim3((unsigned)((nthr + 255) / 256)), dim3(256), 0, stream, p,
                     reinterpret_cast<const T*>(wk.dBp), reinterpret_cast<const T*>(wk.dCp), nrows, R * nmb,
                     (int64_t)p.Bsz * p.L * p.H * p.N);
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
