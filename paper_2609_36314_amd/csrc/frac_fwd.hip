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
// per-mode log-decays l_{t,m} (the log-space form of the appendix: chunk-local sums
// of the capped exponents r_m dtt, in float64; frac_device.h), never from a ratio of
// sequence-global products, so it is exact for any mix of effective steps.
//
// Kernels:
//   frac_cb_kernel   G_chunk = C B^T (Q x Q, causal 16x16 tiles) once per
//                    (batch, chunk, group) -- shared by every head of the group --
//                    stored in the per-lane fragment order the scan reads back.
//   frac_fwd_kernel  one workgroup of 8 waves per (batch, head), or two per
//                    (batch, head) splitting the columns of P when there are 8
//                    modes or too few heads to fill the chip.  Each wave owns a
//                    16-column block of P and either a share of the modes (two or
//                    more modes; it then holds all N rows of its modes) or half of
//                    N (one mode).  Its share of the float32 M x N x P state lives
//                    in matrix-core accumulator registers for the whole sequence
//                    and never touches memory.  Per chunk: x, B and C are copied
//                    straight into LDS (double-buffered for bfloat16, the next
//                    chunk's copy in flight during this chunk's products);
//                    per-token controls and per-(token, mode) weights (lane =
//                    token); (G o Gamma) tiles split over the waves; readout,
//                    intra-chunk product and state update as 16x16x32 matrix-core
//                    products (bfloat16 operands, float32 accumulation).  The
//                    accumulator tiles of the state are converted in registers
//                    straight into B operands of the readout: their row order
//                    becomes the K-slot order, matched by the order in which C is
//                    read from LDS.  Waves that split the modes add their partial
//                    outputs through LDS exchange slots before y is stored.
//                    A state-only instance scans the segments of a split sequence
//                    to their end states (frac_seg_combine_kernel chains them into
//                    boundary states); a mode-block instance covers eight modes of
//                    a larger bank, its weights normalised over the whole bank
//                    (frac_mode_lse_kernel), its outputs summed in float32.
//
// Gamma uses the factorised form (c e^{-r A_t}) (kappa e^{r A_k}) through a float32
// 16x16x4 product with the modes as K, for every mode whose chunk decay r_m A_Q
// stays below 55 (so e^{r A_k} cannot overflow); other modes fall back to one exp
// per (t, k) pair.  The per-mode decay of the state is not applied to the
// accumulators every chunk: the state is held as E_m * S^_m with a float scale E_m
// that absorbs the chunk decays, and the accumulators are rescaled only when E_m
// would fall below 2^-60.
#include <algorithm>

#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

// lower-triangular 16x16 tiles of the Q x Q matrix: (row block, column block)
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
    const int tb = tile_row(tile), kb = tile_col(tile);
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

// LDS row strides (elements) of the staged tiles, padded so that the transposed
// fragment reads of 4 consecutive rows and the row reads of 16 rows spread over
// the LDS banks.  bfloat16 tiles are double-buffered: the next chunk is copied
// in (direct global -> LDS) while the current one is computed.  The block is
// always 8 waves: 4 blocks of 16 columns of P times 2 parts.
template <typename T, int MP, int NB, int PS_ = (MP >= 8 ? 2 : 1), bool SO = false>
struct FwdCfg {
  static constexpr int NP = NB * 16;
  static constexpr bool kBf16 = sizeof(T) == 2;
  static constexpr int XS = kBf16 ? 64 + 8 : 64 + 4;    // x tile   [t][p]
  static constexpr int BS = kBf16 ? NP + 16 : NP + 8;   // B tile   [t][n]
  static constexpr int CS = kBf16 ? NP + 8 : NP + 4;    // C tile   [t][n]
  static constexpr int GS = kBf16 ? 64 + 8 : 64 + 4;    // ((C B^T) o Gamma)^T [k][t]
  static constexpr int NBUF = kBf16 ? 2 : 1;
  // Two waves per 16-column block of P.  With two or more modes they split the
  // modes (each holds all of N for its modes); with one mode they split N.
  // With 8 modes the columns of P are split over two workgroups (PS) so that
  // every wave holds at most 2 modes x all of N of state.  The 8 waves of a
  // workgroup are NPW blocks of 16 columns of P times NPART parts; the parts
  // split the modes (2 or more modes) or N (one mode).  The state-only pass (SO)
  // has no outputs to exchange and splits the modes first, then N.
  static constexpr int PS = PS_;
  static constexpr int NPW = 4 / PS;
  static constexpr bool kModeSplit = MP >= 2;
  static constexpr int NPARTS = 8 / NPW;  // waves per 16-column block of P
  static constexpr int NPM = SO ? (MP < NPARTS ? MP : NPARTS) : (kModeSplit ? NPARTS : 1);  // mode groups
  static constexpr int NPN = SO ? (NPARTS / NPM < NB ? NPARTS / NPM : NB)
                                : (kModeSplit ? 1 : (NB >= 2 ? 2 : 1));  // N groups
  static constexpr int NPART = NPM * NPN;
  static constexpr int MPW = MP / NPM;   // modes per wave
  static constexpr int NBW = NB / NPN;   // 16-row blocks of N per wave
  static constexpr int KBW = (NBW + 1) / 2;                           // 32-deep K steps of the readout
  static constexpr int TBO = 4 / NPART;                               // row blocks of y finished per wave
  // row blocks of the readout whose C fragments are held at once (register budget)
  static constexpr int TBP = (kBf16 ? MPW * NBW < 16 : MPW * NBW < 8) ? 4 : (kBf16 || MPW * NBW < 16) ? 2 : 1;
};

// STATE_ONLY: only the state update over one sequence segment (all but the last),
// from a zero state (the first segment: the initial state), ending in that
// segment's slot of seg_state, with the segment's per-mode decay (the first pass
// of a sequence-split forward).
// BLK: one block of a mode-block launch sequence (weights normalised with p.lse,
// outputs accumulated through p.y_in / p.y_part).
// The state-only pass allocates no C, output or Gamma tiles and is held to 128
// registers, so that two of its workgroups share a CU.
template <typename T, int MP, int NB, int PS, bool STATE_ONLY, bool BLK = false>
__global__ void __launch_bounds__(512, STATE_ONLY ? 4 : 1) frac_fwd_kernel(ScanParams p, const T* __restrict__ gtiles) {
  using Cfg = FwdCfg<T, MP, NB, PS, STATE_ONLY>;
  constexpr int NP = Cfg::NP, XS = Cfg::XS, BS = Cfg::BS, CS = Cfg::CS, GS = Cfg::GS;
  constexpr int NPART = Cfg::NPART, MPW = Cfg::MPW, NBW = Cfg::NBW, KBW = Cfg::KBW, TBP = Cfg::TBP;
  constexpr int NWT = 8;                  // waves in the workgroup
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  // Sequence segment: with p.nseg > 1 the grid holds the (batch, head) blocks once
  // per segment (the state-only pass: per segment but the last), segment k covering
  // tokens [k seg_len, (k + 1) seg_len).
  const int nbh_blocks = p.Bsz * p.H * Cfg::PS;
  const int seg = p.nseg > 1 ? (int)blockIdx.x / nbh_blocks : 0;
  const int bid = (int)blockIdx.x - seg * nbh_blocks;
  const int ps = bid % Cfg::PS;                         // which columns of P
  const int pb = ps * Cfg::NPW + wave % Cfg::NPW, part = wave / Cfg::NPW;
  // waves past the P blocks (or the second part when there is one) only stage
  // tiles, compute controls and Gamma tiles
  const bool active = pb * 16 < p.PP && part < NPART;
  const int mo = (part % Cfg::NPM) * MPW;   // first mode of this wave
  const int nbo = (part / Cfg::NPM) * NBW;  // first N block of this wave
  const int pc = pb * 16 + li;
  const int L = p.L, H = p.H, P = p.P, N = p.N, M = p.M, G = p.G;
  const int Ps = p.Pst;  // row stride of x, y and the P extent of the states
  const int nchunks = (L + kQ - 1) / kQ;
  const int T0 = seg * p.seg_len;                                                // first token
  const int T1 = p.nseg > 1 ? min(L, (seg + 1) * p.seg_len) : L;                // one past the last
  const int c0 = T0 / kQ, c1 = (T1 + kQ - 1) / kQ;                              // chunks of the segment
  const int64_t seg_ss = (int64_t)p.Bsz * p.H * p.Mall * p.N * Ps;              // one boundary state
  const float* init_state = seg == 0 ? p.init_state : (STATE_ONLY ? nullptr : p.seg_state + (seg - 1) * seg_ss);
  float* final_state = STATE_ONLY ? p.seg_state + seg * seg_ss : (T1 == L ? p.final_state : nullptr);
  double seg_ell = 0.0;  // state-only pass, thread m < M: the segment's summed log-decay of mode m

  // Blocks are dealt round-robin to the 8 XCDs; give each XCD a contiguous run of
  // (batch, head) so that heads sharing B and C share one L2.
  int j = bid / Cfg::PS;
  const int nblk = nbh_blocks / Cfg::PS;
  if ((nblk & 7) == 0) j = (j & 7) * (nblk >> 3) + (j >> 3);
  const int b = j / H, h = j - b * H, g = h * G / H;

  __shared__ __align__(16) T Xb0[64 * XS], Bb0[64 * BS], Cb0[STATE_ONLY ? 8 : 64 * CS];
  __shared__ __align__(16) T Xb1[Cfg::NBUF == 2 ? 64 * XS : 8], Bb1[Cfg::NBUF == 2 ? 64 * BS : 8],
      Cb1[Cfg::NBUF == 2 && !STATE_ONLY ? 64 * CS : 8];
  // everything else in one array, so that its addresses differ by constants
  constexpr int oGG = 0;                                        // T [64][GS] ((C B^T) o Gamma)^T, causal
  constexpr int oYb = oGG + (STATE_ONLY ? 0 : 64 * GS * (int)sizeof(T));           // T [64][XS] output rows of the previous chunk
  constexpr int oPrm = oYb + (STATE_ONLY ? 0 : 64 * XS * (int)sizeof(T));          // float [8 MP][Q] per-token weights, log-decays
  constexpr int NSLOT = 4 - Cfg::TBO;                           // row blocks a wave hands over
  constexpr int oYX = oPrm + 8 * MP * kWQ * 4;                  // float [8 waves][NSLOT][4][64] readout exchange
  constexpr int oSc = oYX + (NPART > 1 && !STATE_ONLY ? 8 * NSLOT * 256 : 4) * 4;  // float rates, log tau, scales
  __shared__ __align__(16) unsigned char sm[oSc + 4 * MP * 4];
  T* GGT = reinterpret_cast<T*>(sm + oGG);
  T* Yb = reinterpret_cast<T*>(sm + oYb);
  float* prm = reinterpret_cast<float*>(sm + oPrm);
  float* YX = reinterpret_cast<float*>(sm + oYX);
  float* s_rr = reinterpret_cast<float*>(sm + oSc);
  float* s_lnt = s_rr + MP;
  float* s_E2 = s_lnt + MP;  // [2][MP] by chunk parity
  float* P_om = prm;              // [MP][Q] c e^{-rA_t} E_m        (readout)
  float* P_v = P_om + MP * kWQ;    // [MP][Q] kappa e^{-r(A_Q-A_t)} upd (update)
  float* P_O = P_v + MP * kWQ;     // [MP][Q] c e^{-r A_t}            (Gamma rows)
  float* P_Vt = P_O + MP * kWQ;    // [MP][Q] kappa e^{r A_t}, safe modes (Gamma columns)
  float* P_c = P_Vt + MP * kWQ;    // [MP][Q] c      (modes past the factorisation bound)
  float* P_k = P_c + MP * kWQ;     // [MP][Q] kappa
  float* P_lh = P_k + MP * kWQ;    // [MP][Q] chunk log-decays l_{t,m}, hi and lo parts
  float* P_ll = P_lh + MP * kWQ;

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * Ps;
  const T* Bgp = reinterpret_cast<const T*>(p.Bm) + (((int64_t)b * L) * G + g) * N;
  const T* Cgp = reinterpret_cast<const T*>(p.Cm) + (((int64_t)b * L) * G + g) * N;
  T* yg = reinterpret_cast<T*>(p.y) + (((int64_t)b * L) * H + h) * Ps;
  const int64_t xstride = (int64_t)H * Ps, bstride = (int64_t)G * N;

  // per-mode rates 1/tau_m, log tau_m and state scales E_m (by chunk parity) in LDS
  if (tid < MP) {
    const float tau = (tid < M) ? p.tau[tid] : 1.0f;
    s_rr[tid] = (tid < M) ? 1.0f / tau : 0.0f;
    s_lnt[tid] = (tid < M) ? logf(tau) : 0.0f;
    s_E2[tid] = s_E2[MP + tid] = 1.0f;
  }
  // tiles start zeroed: columns past P or N are never copied into
  if constexpr (!STATE_ONLY)
    for (int i = tid; i < 64 * GS; i += 512) GGT[i] = (T)0.0f;
  for (int i = tid; i < 64 * XS; i += 512) Xb0[i] = Xb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;
  for (int i = tid; i < 64 * BS; i += 512) Bb0[i] = Bb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;
  if constexpr (!STATE_ONLY)
    for (int i = tid; i < 64 * CS; i += 512) Cb0[i] = Cb1[Cfg::NBUF == 2 ? i : 0] = (T)0.0f;

  // ---- state: S[m][jb] holds mode mo + m, rows n = 16 (nbo + jb) + 4 lg + r, column pc
  const int64_t sbase = ((int64_t)b * H + h) * (int64_t)p.Mall * N * Ps;
  floatx4 S[MPW][NBW];
  {
    // lane offset kept opaque so that the final store cannot share (and keep alive
    // across the sequence loop) the per-element offsets of this load
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
          if (init_state && active && mo + m < M && n < N && pc < P)
            v = init_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * Ps];
          S[m][jb][r] = v;
        }
  }
  const float Dh = p.D ? p.D[h] : 0.0f;

  // per-token controls of a chunk, loaded one chunk ahead (lane = token)
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const int64_t al_st = p.as1;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const int64_t lm_st = p.ls1;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * p.Mall : nullptr;
  const bool w_is_c = wl_bh == rl_bh;  // then the write weights equal the read weights
  const int64_t lg_st = (int64_t)H * p.Mall;
  const float* lse_bh = BLK ? p.lse + ((int64_t)b * L * H + h) * 2 : nullptr;  // [t][H][2]
  PairLogits<MP, 512, BLK> lgt_n;  // the logits (and normalizers) of the next chunk's weight pass
  auto load_controls = [&](int c, float& dtv, float& al, float& lam) {
    const int tg = c * kQ + lane;
    const bool valid = tg < T1;
    dtv = valid ? dt_bh[(int64_t)tg * H] : 0.0f;
    al = valid ? al_bh[tg * al_st] : 1.0f;
    lam = (valid && lm_bh) ? lm_bh[tg * lm_st] : 1.0f;
    lgt_n.load(rl_bh, wl_bh, c * kQ, min(kQ, T1 - c * kQ), M, lg_st, tid, lse_bh, (int64_t)H * 2);
  };
  DmaPlan<T, XS> planX;
  DmaPlan<T, BS> planB;
  DmaPlan<T, CS> planC;
  planX.init(xstride, P);
  planB.init(bstride, N);
  planC.init(bstride, N);
  auto stage = [&](int c, T* Xd, T* Bd, T* Cd) {
    const int t0 = c * kQ, nv = min(kQ, T1 - t0);
    planX.issue_async(Xd, xg + (int64_t)t0 * xstride, xstride, nv);
    planB.issue_async(Bd, Bgp + (int64_t)t0 * bstride, bstride, nv);
    if constexpr (!STATE_ONLY) planC.issue_async(Cd, Cgp + (int64_t)t0 * bstride, bstride, nv);
  };
  // output rows of chunk c (staged in Yb) -> global, 16 bytes per thread
  auto store_y = [&](int c) {
    constexpr int E8 = 16 / sizeof(T);
    const int t0 = c * kQ, nv = min(kQ, T1 - t0);
    constexpr int CY = 64 / E8;  // 16-byte chunks of a 64-column row
#pragma unroll
    for (int i0 = 0; i0 < 64 * CY; i0 += 512) {
      const int i = i0 + tid, t = i / CY, ch = i & (CY - 1);
      const int col = ch * E8;  // only this workgroup's columns of P
      if (t < nv && col < P && col >= ps * Cfg::NPW * 16 && col < (ps + 1) * Cfg::NPW * 16)
        *reinterpret_cast<int4*>(yg + (int64_t)(t0 + t) * xstride + ch * E8) =
            *reinterpret_cast<const int4*>(Yb + t * XS + ch * E8);
    }
  };

  float dt_n, al_n, lam_n;
  load_controls(c0, dt_n, al_n, lam_n);
  TilePrefetch<T> gtile;  // C B^T tile values, loaded one chunk ahead
  if constexpr (!STATE_ONLY)
    gtile.load(gtiles + (((int64_t)b * nchunks + c0) * G + g) * (kTiles * kTileElems), wave, lane);
  if (Cfg::NBUF == 2) stage(c0, Xb0, Bb0, Cb0);

  // one chunk: Xc/Bc/Cc hold it (or receive it when single-buffered), Xn/Bn/Cn
  // receive the next one
  auto step = [&](int c, T* Xc, T* Bc, T* Cc, T* Xn, T* Bn, T* Cn) __attribute__((always_inline)) {
    const int t0 = c * kQ;
    const int nv = min(kQ, T1 - t0);
    const float* Ecur = s_E2 + (c & 1) * MP;
    float* Enext = s_E2 + ((c + 1) & 1) * MP;
    wait_vmem();
    barrier();  // this chunk's tiles have landed; every wave is done with the previous chunk
    // this chunk's prefetched controls, logits and C B^T values, taken before any new memory operation
    const float dtv = pinned(dt_n), al_l = pinned(al_n), lam_l = pinned(lam_n);
    const PairLogits<MP, 512, BLK> lgt = lgt_n.pinned_copy();
    const TilePrefetch<T> gcur = gtile.pinned_copy();
    if (!STATE_ONLY && c > c0 && !(BLK && p.y_part)) store_y(c - 1);
    if (Cfg::NBUF == 2) {
      if (c + 1 < c1) stage(c + 1, Xn, Bn, Cn);
    } else {
      stage(c, Xc, Bc, Cc);
      wait_vmem();
      barrier();
    }
    if (c + 1 < c1) load_controls(c + 1, dt_n, al_n, lam_n);

    // ---- per-token step (lane = token, every wave) and the per-mode log-decays
    const float s_eff_l = lm_bh ? step_factor(lam_l, al_l) : 1.0f;
    const float dtt_l = (lane < nv) ? dtv * s_eff_l : 0.0f;
    chunk_log_decays<MP, NWT>(dtt_l, s_rr, P_lh, P_ll);
    barrier();  // log-decays in LDS
    if (STATE_ONLY && tid < MP) seg_ell += (double)P_lh[tid * kWQ + kQ - 1] + (double)P_ll[tid * kWQ + kQ - 1];

    // ---- per (token, mode) controls and weights: thread pair = t MP + m
    // bit m of unsafe: the factorised Gamma would overflow for mode m (direct decay);
    // the same flags in every wave, lane m < MP testing mode m
    const bool over = lane < MP && lane < M && !(P_lh[(lane < MP ? lane : 0) * kWQ + kQ - 1] <= kSafeExponent);
    const int unsafe = (int)(__ballot(over) & ((1ull << MP) - 1));
#pragma unroll
    for (int j = 0; j < lgt.NPR; ++j) {
      const int pr = tid + 512 * j;
      if (pr >= kQ * MP) break;  // wave-uniform
      const int t = pr / MP, m = pr - t * MP;
      const float dtt = __shfl(dtt_l, t, 64), al = __shfl(al_l, t, 64);
      const bool valid = t < nv;
      const float r = s_rr[m], prior = -al * s_lnt[m];
      float zc = (m < M) ? prior + lgt.rl[j] : -INFINITY;
      float zw = (m < M) ? prior + lgt.wl[j] : -INFINITY;
      // tokens past the sequence get zero weights (their tile rows may hold anything finite);
      // a mode block normalises over all modes with the precomputed log-normalizers
      const float lhQ = P_lh[m * kWQ + kQ - 1];
      const float Enew = Ecur[m] * fexp(-lhQ);
      const bool ren = !(Enew >= kRescaleFloor);
      const float upd = ren ? 1.0f : fast_rcp(Enew);
      if constexpr (STATE_ONLY) {  // the state update only: the write weights
        float ww;
        if constexpr (BLK) {
          const float ln = w_is_c ? __shfl(lgt.ln_c, t, 64) : __shfl(lgt.ln_w, t, 64);
          ww = valid ? __expf((w_is_c ? zc : zw) - ln) : 0.0f;
        } else {
          ww = valid ? group_softmax<MP>(w_is_c ? zc : zw) : 0.0f;
        }
        const float kap = one_minus_exp_neg(dtt * r) * ww;
        P_v[m * kWQ + t] = kap * ell_decay(P_lh + m * kWQ, P_ll + m * kWQ, kQ - 1, t) * upd;
      } else {
        float cw, ww;
        if constexpr (BLK) {
          const float lnc = __shfl(lgt.ln_c, t, 64), lnw = __shfl(lgt.ln_w, t, 64);
          cw = valid ? __expf(zc - lnc) : 0.0f;
          ww = w_is_c ? cw : (valid ? __expf(zw - lnw) : 0.0f);
        } else {
          cw = valid ? group_softmax<MP>(zc) : 0.0f;
          ww = w_is_c ? cw : (valid ? group_softmax<MP>(zw) : 0.0f);
        }
        const float lh = P_lh[m * kWQ + t];
        const bool safe = lhQ <= kSafeExponent;
        const float kap = one_minus_exp_neg(dtt * r) * ww;
        const float om = cw * fexp(-lh);
        P_O[m * kWQ + t] = om;
        P_om[m * kWQ + t] = om * Ecur[m];
        P_v[m * kWQ + t] = kap * ell_decay(P_lh + m * kWQ, P_ll + m * kWQ, kQ - 1, t) * upd;
        P_Vt[m * kWQ + t] = safe ? kap * fexp(lh) : 0.0f;
        P_c[m * kWQ + t] = cw;
        P_k[m * kWQ + t] = kap;
      }
      if (pr < MP) Enext[m] = ren ? 1.0f : Enew;
    }
    // this wave's modes: rescale flags and factors (wave-uniform)
    float renf[MPW];
    int renbits = 0;
#pragma unroll
    for (int m = 0; m < MPW; ++m) {
      const float Enew = uniform(Ecur[mo + m] * fexp(-P_lh[(mo + m) * kWQ + kQ - 1]));
      renf[m] = Enew;
      if (__float_as_int(Enew) < __float_as_int(kRescaleFloor)) renbits |= 1 << m;
    }
    barrier();  // controls in LDS
    if constexpr (!STATE_ONLY) {

    __builtin_amdgcn_sched_barrier(0);
    // ---- ((C B^T) o Gamma)^T, lower-triangular 16x16 tiles split over the waves
    {
#pragma unroll
      for (int jt = 0; jt < 2; ++jt) {
        const int tile = wave + NWT * jt;
        if (tile >= kTiles) break;
        const int tb = tile_row(tile), kb = tile_col(tile);
        float Gt[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) Gt[r] = gcur.get(jt, r);
        floatx4 Gm = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < (MP + 3) / 4; ++q) {
          const int m = q * 4 + lg;
          const float av = (m < MP) ? P_O[m * kWQ + tb * 16 + li] : 0.0f;
          const float bv = (m < MP) ? P_Vt[m * kWQ + kb * 16 + li] : 0.0f;
          Gm = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, Gm, 0, 0, 0);
        }
        if (unsafe) {
          for (int m = 0; m < MP; ++m) {
            if (!((unsafe >> m) & 1)) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
              if (t >= k) Gm[r] += P_c[m * kWQ + t] * P_k[m * kWQ + k] * ell_decay(P_lh + m * kWQ, P_ll + m * kWQ, t, k);
            }
          }
        }
        float gv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
          gv[r] = keep_if_ge(Gt[r] * Gm[r], t, k);
        }
        T* dst = GGT + (kb * 16 + li) * GS + tb * 16 + lg * 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[r] = (T)gv[r];
      }
    }

    if (c + 1 < c1) gtile.load(gtiles + (((int64_t)b * nchunks + c + 1) * G + g) * (kTiles * kTileElems), wave, lane);

    __builtin_amdgcn_sched_barrier(0);
    // ---- readout of the state entering the chunk, this wave's modes
    floatx4 Y[4];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) Y[tb] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (active) {
#pragma unroll
    for (int tp = 0; tp < 4 / TBP; ++tp) {
      Frag<T> Ca[TBP][KBW];
#pragma unroll
      for (int i = 0; i < TBP; ++i)
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          const T* row = Cc + ((tp * TBP + i) * 16 + li) * CS + nbo * 16 + kb * 32 + lg * 4;
          Ca[i][kb] = frag_load4x2(row, row + 16, 2 * kb + 1 < NBW);
        }
#pragma unroll
      for (int m = 0; m < MPW; ++m) {
        Frag<T> Sf[KBW];  // modes >= M hold a zero state and zero weights
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Sf[kb], s, S[m][2 * kb][s]);
#pragma unroll
          for (int s = 0; s < 4; ++s) frag_set(Sf[kb], 4 + s, (2 * kb + 1 < NBW) ? S[m][2 * kb + 1][s] : 0.0f);
        }
#pragma unroll
        for (int i = 0; i < TBP; ++i) {
          const int tb = tp * TBP + i;
          floatx4 Z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) mma(Z, Ca[i][kb], Sf[kb]);
          const float4 om = *reinterpret_cast<const float4*>(P_om + (mo + m) * kWQ + tb * 16 + lg * 4);
          Y[tb][0] += om.x * Z[0];
          Y[tb][1] += om.y * Z[1];
          Y[tb][2] += om.z * Z[2];
          Y[tb][3] += om.w * Z[3];
        }
      }
    }
    if (NPART > 1) {
      // hand the row blocks the other parts of this P block finish over through LDS
      float* dst = YX + wave * NSLOT * 256;
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        if (tb / Cfg::TBO == part) continue;
        const int slot = tb < part * Cfg::TBO ? tb : tb - Cfg::TBO;
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[(slot * 4 + r) * 64 + lane] = Y[tb][r];
      }
    }
    }  // active
    barrier();  // GGT and YX complete
    if (!active) return;

    __builtin_amdgcn_sched_barrier(0);
    // ---- intra-chunk product, skip term, output rows into Yb
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      if (NPART > 1 && tb / Cfg::TBO != part) continue;
      // partial sums of the other parts, added in part order
#pragma unroll
      for (int q = 0; q < NPART; ++q) {
        if (q == part) continue;
        const int slot = tb < q * Cfg::TBO ? tb : tb - Cfg::TBO;
        const float* src = YX + (q * Cfg::NPW + wave % Cfg::NPW) * NSLOT * 256;
#pragma unroll
        for (int r = 0; r < 4; ++r) Y[tb][r] += src[(slot * 4 + r) * 64 + lane];
      }
#pragma unroll
      for (int kk = 0; kk <= tb / 2; ++kk) {
        const Frag<T> a = frag_load_rows(GGT, GS, kk * 32 + lg * 8, tb * 16);
        const Frag<T> bb = frag_load_rows(Xc, XS, kk * 32 + lg * 8, pb * 16);
        mma(Y[tb], a, bb);
      }
      float xv[4];
      col4_rows(Xc, XS, tb * 16 + lg * 4, pb * 16, xv);
      if constexpr (BLK) {  // a mode block: float32 partial sums across the blocks
        // one 64-bit base per row block and 32-bit row offsets (per-element 64-bit
        // indices spilled 32 registers here); the four loads issue before any is used
        const int64_t y0 = (((int64_t)b * L + t0 + tb * 16 + lg * 4) * H + h) * Ps + pc;
        const int rs = H * Ps;
        const float* yq = p.y_in;
        float* yp = p.y_part;
        float yv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tr = tb * 16 + lg * 4 + r;
          yv[r] = (yq && tr < nv && pc < P) ? yq[y0 + r * rs] : 0.0f;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tr = tb * 16 + lg * 4 + r;
          Y[tb][r] += yv[r];
          if (yp && tr < nv && pc < P) yp[y0 + r * rs] = Y[tb][r];
        }
      }
      if (!(BLK && p.y_part)) {
#pragma unroll
        for (int r = 0; r < 4; ++r) Yb[(tb * 16 + lg * 4 + r) * XS + pc] = (T)(Y[tb][r] + Dh * xv[r]);
      }
    }
    }  // !STATE_ONLY
    if (!active) return;

    __builtin_amdgcn_sched_barrier(0);
    // ---- state update  S_m <- (rescale) + B^T (v_m o X), this wave's modes
#pragma unroll
    for (int m = 0; m < MPW; ++m) {
      if (!((renbits >> m) & 1)) continue;
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) S[m][jb][r] *= renf[m];
    }
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const Frag<T> xf = frag_load_rows(Xc, XS, kt * 32 + lg * 8, pb * 16);
      Frag<T> Xf[MPW];
#pragma unroll
      for (int m = 0; m < MPW; ++m) {
        const float* pv = P_v + (mo + m) * kWQ + kt * 32 + lg * 8;
        const float4 v0 = *reinterpret_cast<const float4*>(pv);
        const float4 v1 = *reinterpret_cast<const float4*>(pv + 4);
        frag_set(Xf[m], 0, to_f32(xf.v[0]) * v0.x);
        frag_set(Xf[m], 1, to_f32(xf.v[1]) * v0.y);
        frag_set(Xf[m], 2, to_f32(xf.v[2]) * v0.z);
        frag_set(Xf[m], 3, to_f32(xf.v[3]) * v0.w);
        frag_set(Xf[m], 4, to_f32(xf.v[4]) * v1.x);
        frag_set(Xf[m], 5, to_f32(xf.v[5]) * v1.y);
        frag_set(Xf[m], 6, to_f32(xf.v[6]) * v1.z);
        frag_set(Xf[m], 7, to_f32(xf.v[7]) * v1.w);
      }
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb) {
        const Frag<T> a = frag_load_rows(Bc, BS, kt * 32 + lg * 8, (nbo + jb) * 16);
#pragma unroll
        for (int m = 0; m < MPW; ++m)
          mma(S[m][jb], a, Xf[m]);  // modes >= M carry zero weights
      }
    }
  };

  for (int c = c0; c < c1; c += 2) {
    step(c, Xb0, Bb0, Cb0, Xb1, Bb1, Cb1);
    if (c + 1 < c1) {
      if (Cfg::NBUF == 2) step(c + 1, Xb1, Bb1, Cb1, Xb0, Bb0, Cb0);
      else step(c + 1, Xb0, Bb0, Cb0, Xb0, Bb0, Cb0);
    }
  }
  wait_vmem();
  barrier();
  if (!STATE_ONLY && !(BLK && p.y_part)) store_y(c1 - 1);
  if (STATE_ONLY && ps == 0 && tid < M)
    p.seg_decay[((int64_t)seg * p.Bsz * H + (int64_t)b * H + h) * p.Mall + tid] = (float)exp(-seg_ell);

  if (final_state && active) {
    const float* Ef = s_E2 + (c1 & 1) * MP;
    int lo = (mo * N + nbo * 16 + lg * 4) * Ps + pc;
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int m = 0; m < MPW; ++m) {
      const float Em = (mo + m < M) ? Ef[mo + m] : 0.0f;
#pragma unroll
      for (int jb = 0; jb < NBW; ++jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = (nbo + jb) * 16 + lg * 4 + r;
          if (mo + m < M && n < N && pc < P)
            final_state[sbase + lo + ((int64_t)m * N + jb * 16 + r) * Ps] = S[m][jb][r] * Em;
        }
    }
  }
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

// Workgroups per (batch, head) along P: two with 8 modes (register budget); with 4
// modes two when few (batch, head) pairs would leave compute units idle and the
// sequence is too short to split.
int fwd_p_split(const ScanParams& p) {
  const int MP = p.M <= 1 ? 1 : p.M <= 2 ? 2 : p.M <= 4 ? 4 : 8;
  const int nchunks = (p.L + kQ - 1) / kQ;
  return (MP >= 8 || (MP >= 4 && p.Bsz * p.H < 192 && nchunks < 16)) ? 2 : 1;
}

// Sequence split: when the (batch, head) workgroups fill fewer than two per compute
// unit (512) and the sequence is long, it is cut into up to 16 segments of whole
// chunks (at least 4 each).  A state-only pass scans every segment but the last
// from a zero state, a combine pass chains their end states into the boundary
// states, and the output pass runs all segments at once.
struct FwdSplit {
  int nseg, seg_len;
};

FwdSplit fwd_split(const ScanParams& p) {
  const int nchunks = (p.L + kQ - 1) / kQ;
  const int64_t wg = (int64_t)p.Bsz * p.H * fwd_p_split(p);
  if (wg >= 512 || nchunks < 8) return {1, p.L};
  int k = (int)std::min<int64_t>({(int64_t)16, (512 + wg - 1) / wg, (int64_t)(nchunks / 4)});
  if (k < 2) return {1, p.L};
  const int per = (nchunks + k - 1) / k;
  return {(nchunks + per - 1) / per, per * kQ};
}

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Boundary states and decays of a split forward, after the C B^T tiles.
size_t split_bytes(const ScanParams& p, const FwdSplit& sp) {
  if (sp.nseg <= 1) return 0;
  const size_t ns = (size_t)sp.nseg - 1, bhm = (size_t)p.Bsz * p.H * p.Mall;
  return align256(sizeof(float) * ns * bhm * p.N * p.Pst) + align256(sizeof(float) * ns * bhm);
}

void place_split(ScanParams& p, const FwdSplit& sp, unsigned char* at) {
  p.nseg = sp.nseg;
  p.seg_len = sp.seg_len;
  if (sp.nseg <= 1) {
    p.seg_state = nullptr;
    p.seg_decay = nullptr;
    return;
  }
  const size_t ns = (size_t)sp.nseg - 1, bhm = (size_t)p.Bsz * p.H * p.Mall;
  p.seg_state = reinterpret_cast<float*>(at) + p.col0;  // this column group's columns
  p.seg_decay = reinterpret_cast<float*>(at + align256(sizeof(float) * ns * bhm * p.N * p.Pst));
}

// The boundary states: S_k = decay_k S_{k-1} + (segment k's own end state), in
// segment order, per state element (all modes of the bank, this column group's P).
__global__ void __launch_bounds__(256) frac_seg_combine_kernel(ScanParams p) {
  const int64_t ss = (int64_t)p.Bsz * p.H * p.Mall * p.N * p.Pst;  // one boundary state
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)p.Bsz * p.H * p.Mall * p.N * p.P) return;
  const int64_t row = i / p.P, e = row * p.Pst + (i - row * p.P);  // (b, h, m, n) row, column
  const int64_t bhm = row / p.N, nbhm = (int64_t)p.Bsz * p.H * p.Mall;
  float s = p.seg_state[e];
  for (int k = 1; k + 1 < p.nseg; ++k) {
    s = p.seg_decay[k * nbhm + bhm] * s + p.seg_state[k * ss + e];
    p.seg_state[k * ss + e] = s;
  }
}

hipError_t launch_seg_combine(const ScanParams& p, hipStream_t stream) {
  if (p.nseg <= 2) return hipSuccess;  // one boundary: the first segment's end state
  const int64_t n = (int64_t)p.Bsz * p.H * p.Mall * p.N * p.P;
  hipLaunchKernelGGL(frac_seg_combine_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

// The state-only pass over every segment but the last (one workgroup per (batch,
// head) and PS column blocks, as the output pass).
template <typename T, int MP, int NB, int PS, bool BLK = false>
hipError_t launch_fwd_state_pass(const ScanParams& p, const T* gt, hipStream_t stream) {
  if (p.nseg <= 1) return hipSuccess;
  const unsigned blocks = (unsigned)(p.Bsz * p.H * PS * (p.nseg - 1));
  hipLaunchKernelGGL((frac_fwd_kernel<T, MP, NB, PS, true, BLK>), dim3(blocks), dim3(512), 0, stream, p, gt);
  return hipGetLastError();
}

template <typename T, int MP, int NB, int PS, bool BLK = false>
hipError_t launch_fwd_out_pass(const ScanParams& p, const T* gt, hipStream_t stream) {
  const unsigned blocks = (unsigned)(p.Bsz * p.H * PS * p.nseg);
  hipLaunchKernelGGL((frac_fwd_kernel<T, MP, NB, PS, false, BLK>), dim3(blocks), dim3(512), 0, stream, p, gt);
  return hipGetLastError();
}

template <typename T, int MP, int NB, int PS>
hipError_t launch_fwd_ps(const ScanParams& p, const T* gt, hipStream_t stream) {
  hipError_t e = launch_fwd_state_pass<T, MP, NB, PS>(p, gt, stream);
  if (e == hipSuccess) e = launch_seg_combine(p, stream);
  if (e == hipSuccess) e = launch_fwd_out_pass<T, MP, NB, PS>(p, gt, stream);
  return e;
}

template <typename T, int MP, int NB>
hipError_t launch_fwd_variant(const ScanParams& p0, void* ws, hipStream_t stream) {
  T* gt = reinterpret_cast<T*>(ws);
  hipError_t e = launch_cb_variant<T, NB>(p0, gt, stream);
  if (e != hipSuccess) return e;
  ScanParams p = p0;
  place_split(p, fwd_split(p), reinterpret_cast<unsigned char*>(ws) + align256(gtile_bytes<T>(p)));
  if constexpr (MP >= 8) return launch_fwd_ps<T, MP, NB, 2>(p, gt, stream);
  else if constexpr (MP >= 4) {
    if (fwd_p_split(p) == 2) return launch_fwd_ps<T, MP, NB, 2>(p, gt, stream);
    return launch_fwd_ps<T, MP, NB, 1>(p, gt, stream);
  } else {
    return launch_fwd_ps<T, MP, NB, 1>(p, gt, stream);
  }
}

// Per token (b, t, h): the log-normalizers of the read and write softmax over all
// Mall modes, z_m = -alpha ln tau_m + logit_m (eq. read-softmax), as max + log sum exp.
__global__ void __launch_bounds__(256) frac_mode_lse_kernel(ScanParams p, float* __restrict__ lse) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)p.Bsz * p.L * p.H) return;
  const int h = (int)(i % p.H);
  const int64_t bt = i / p.H;
  const int t = (int)(bt % p.L), b = (int)(bt / p.L);
  const int Ma = p.Mall;
  const float al = strided3(p.alpha, p.as0, p.as1, p.as2, b, t, h);
  const float* rl = p.read_logit ? p.read_logit + i * Ma : nullptr;
  const float* wl = (p.write_logit && p.write_logit != p.read_logit) ? p.write_logit + i * Ma : nullptr;
  const bool w_is_c = p.write_logit == p.read_logit;
  float mc = -INFINITY, mw = -INFINITY;
  for (int m = 0; m < Ma; ++m) {
    const float prior = -al * logf(p.tau[m]);
    mc = fmaxf(mc, prior + (rl ? rl[m] : 0.0f));
    mw = fmaxf(mw, prior + (wl ? wl[m] : 0.0f));
  }
  float sc = 0.0f, sw = 0.0f;
  for (int m = 0; m < Ma; ++m) {
    const float prior = -al * logf(p.tau[m]);
    sc += __expf(prior + (rl ? rl[m] : 0.0f) - mc);
    sw += __expf(prior + (wl ? wl[m] : 0.0f) - mw);
  }
  const float lc = mc + logf(sc);
  reinterpret_cast<float2*>(lse)[i] = float2{lc, w_is_c ? lc : mw + logf(sw)};
}

constexpr int kModeBlock = 8;  // modes per launch of the mode-block forward

// Workspace of the mode-block forward: [C B^T tiles][boundary state, all modes]
// [log-normalizers][float32 partial output].
struct FwdBlockLayout {
  size_t seg, lse, ypart, total;
  FwdSplit split;
};

template <typename T>
FwdBlockLayout fwd_block_layout(const ScanParams& p) {
  ScanParams pb = p;
  pb.M = kModeBlock;
  FwdBlockLayout l{};
  l.split = fwd_split(pb);
  l.seg = align256(gtile_bytes<T>(p));
  l.lse = l.seg + split_bytes(p, l.split);
  l.ypart = l.lse + align256(sizeof(float) * 2 * (size_t)p.Bsz * p.L * p.H);
  l.total = l.ypart + sizeof(float) * (size_t)p.Bsz * p.L * p.H * p.Pst;
  return l;
}

// More modes than one workgroup's registers hold: the modes in blocks of eight, one
// forward launch per block (the recurrence is linear in the modes once the weights
// are fixed), the weights normalised over all modes, the outputs summed in float32
// in block order; the last block adds the skip term and writes y.
template <typename T, int NB>
hipError_t launch_fwd_blocks(const ScanParams& p0, void* ws, hipStream_t stream) {
  const FwdBlockLayout l = fwd_block_layout<T>(p0);
  unsigned char* base = reinterpret_cast<unsigned char*>(ws);
  T* gt = reinterpret_cast<T*>(ws);
  hipError_t e = launch_cb_variant<T, NB>(p0, gt, stream);
  if (e != hipSuccess) return e;
  float* lse = reinterpret_cast<float*>(base + l.lse);
  float* ypart = reinterpret_cast<float*>(base + l.ypart) + p0.col0;  // this column group's columns
  if ((e = launch_mode_lse(p0, lse, stream)) != hipSuccess) return e;
  const int64_t NP = (int64_t)p0.N * p0.Pst;
  ScanParams ps0 = p0;
  place_split(ps0, l.split, base + l.seg);
  // the state-only passes of every block, the boundary states, then the output passes
  auto block = [&](int mo) {
    ScanParams p = ps0;
    p.M = min(kModeBlock, p0.Mall - mo);
    p.tau = p0.tau + mo;
    if (p0.read_logit) p.read_logit = p0.read_logit + mo;
    if (p0.write_logit) p.write_logit = p0.write_logit + mo;
    if (p0.init_state) p.init_state = p0.init_state + mo * NP;
    if (p0.final_state) p.final_state = p0.final_state + mo * NP;
    p.lse = lse;
    p.y_in = mo > 0 ? ypart : nullptr;
    p.y_part = mo + kModeBlock < p0.Mall ? ypart : nullptr;
    if (p.nseg > 1) {
      p.seg_state = ps0.seg_state + mo * NP;
      p.seg_decay = ps0.seg_decay + mo;
    }
    return p;
  };
  for (int mo = 0; mo < p0.Mall; mo += kModeBlock)
    if ((e = launch_fwd_state_pass<T, kModeBlock, NB, 2, true>(block(mo), gt, stream)) != hipSuccess) return e;
  if ((e = launch_seg_combine(ps0, stream)) != hipSuccess) return e;
  for (int mo = 0; mo < p0.Mall; mo += kModeBlock)
    if ((e = launch_fwd_out_pass<T, kModeBlock, NB, 2, true>(block(mo), gt, stream)) != hipSuccess) return e;
  return hipSuccess;
}

template <typename T, int MP>
hipError_t launch_fwd_nb(const ScanParams& p, void* ws, hipStream_t stream) {
  if constexpr (MP > kModeBlock) {
    switch (p.NP / 16) {
      case 1: return launch_fwd_blocks<T, 1>(p, ws, stream);
      case 2: return launch_fwd_blocks<T, 2>(p, ws, stream);
      case 4: return launch_fwd_blocks<T, 4>(p, ws, stream);
      case 8: return launch_fwd_blocks<T, 8>(p, ws, stream);
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (p.NP / 16) {
      case 1: return launch_fwd_variant<T, MP, 1>(p, ws, stream);
      case 2: return launch_fwd_variant<T, MP, 2>(p, ws, stream);
      case 4: return launch_fwd_variant<T, MP, 4>(p, ws, stream);
      case 8: return launch_fwd_variant<T, MP, 8>(p, ws, stream);
      default: return hipErrorInvalidValue;
    }
  }
}

template <typename T>
hipError_t launch_fwd_mp(const ScanParams& p, void* ws, hipStream_t stream) {
  if (p.M <= 1) return launch_fwd_nb<T, 1>(p, ws, stream);
  if (p.M <= 2) return launch_fwd_nb<T, 2>(p, ws, stream);
  if (p.M <= 4) return launch_fwd_nb<T, 4>(p, ws, stream);
  if (p.M <= 8) return launch_fwd_nb<T, 8>(p, ws, stream);
  return launch_fwd_nb<T, 32>(p, ws, stream);
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

hipError_t launch_mode_lse(const ScanParams& p, float* lse, hipStream_t stream) {
  const int64_t n = (int64_t)p.Bsz * p.L * p.H;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(frac_mode_lse_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, p, lse);
  return hipGetLastError();
}

size_t scan_fwd_workspace(const ScanParams& p) {
  if (p.Bsz == 0 || p.L == 0) return 0;
  if (p.Mall > kModeBlock) return p.io_bf16 ? fwd_block_layout<bf16>(p).total : fwd_block_layout<float>(p).total;
  const size_t tiles = p.io_bf16 ? gtile_bytes<bf16>(p) : gtile_bytes<float>(p);
  return align256(tiles) + split_bytes(p, fwd_split(p));  // + the boundary states and decays
}

hipError_t launch_scan_fwd(const ScanParams& p, void* ws, size_t, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  // headdim above 64: independent groups of 64 columns (the recurrence is per column of P)
  for (int c0 = 0; c0 < p.Pst; c0 += 64) {
    const ScanParams q = column_group(p, c0);
    const hipError_t e = p.io_bf16 ? launch_fwd_mp<bf16>(q, ws, stream) : launch_fwd_mp<float>(q, ws, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace frac
