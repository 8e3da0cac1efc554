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
// The decays are formed from per-mode chunk log-decays l_{t,m} (the chunk-local sums
// of the capped exponents r_m dtt, in float64; frac_device.h), exact for any mix of
// effective steps in a chunk.
//
// One workgroup of NW waves per (batch, head, 16 NW columns of d_h): 8 waves and
// 128 columns for head dims above 128, else 4 and 64; wave w owns columns
// 16 w .. 16 w + 15 and the state of all modes for them (at most two 16x16
// float32 accumulator tiles, modes as rows).  Per chunk: x copied into LDS,
// per-(token, mode) weights, Gamma in causal 16x16 tiles (float32 matrix cores,
// modes as K; one exponential per pair for modes whose chunk decay passes the
// factorisation bound), then the readout (weights x state, K = modes), the
// intra-chunk product Gamma x (K = tokens) and the state update (K = tokens) on
// the matrix cores.  The state scale trick of the B/C scan applies unchanged.
#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

namespace {

typedef unsigned int i32x4_t __attribute__((ext_vector_type(4)));  // a 16-byte buffer access
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));  // an 8-byte buffer access

constexpr float kNfSafe = 55.0f;
constexpr float kNfFloor = 0x1p-60f;


// CKPT: no outputs; the state entering every chunk, and the final state, go to
// ckpt [B H][nchunks + 1][M][P] (the first pass of the backward).  Without CKPT a
// non-NULL ckpt receives the same states beside the outputs (the caller's chunk
// states, which its backward then reads instead of running that pass).
// NW waves per workgroup over 16 NW / NH columns of d_h: with more waves per
// workgroup the per-chunk work that does not depend on the columns (the
// log-decays, the weights, the Gamma tiles) is done once for more columns and
// split over more waves.  With NH = 2 two waves share each 16 columns: both keep
// the state, and each forms the outputs of one half of the chunk's tokens.
// Inside a chunk, global addresses are a wave-uniform chunk base plus 32-bit
// per-lane offsets (the host keeps 64 H d_h below 2^31).
template <typename T, int MP, bool CKPT, int NW = 4, int NH = 1>
__global__ void __launch_bounds__(64 * NW) frac_nfree_fwd_kernel(ScanParams p, float* __restrict__ ckpt) {
  constexpr bool kBf16 = sizeof(T) == 2;
  constexpr int MB = (MP + 15) / 16;        // 16-row blocks of modes in the state
  constexpr int CG = NW / NH;               // 16-column groups (waves per token half)
  constexpr int NT = 64 * NW, CW = 16 * CG;  // threads, columns of d_h per workgroup
  constexpr int XS = kBf16 ? CW + 8 : CW + 4;  // [t][p] tile stride
  constexpr int GS = kBf16 ? 64 + 8 : 64 + 4;  // [t][k] tile stride
  static_assert(NT % MP == 0, "every (token, mode) pair of a thread has the same mode");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int cg = wave % CG, half = wave / CG;  // column group, token half of the readout
  const int L = p.L, H = p.H, P = p.P, M = p.M;
  const int nps = (P + CW - 1) / CW;
  const int ps = blockIdx.x % nps, bh = blockIdx.x / nps, b = bh / H, h = bh - b * H;
  const int p0 = ps * CW, pc = p0 + cg * 16 + li;  // this lane's column of d_h
  const bool active = p0 + cg * 16 < P;
  const int nchunks = (L + kQ - 1) / kQ;

  __shared__ __align__(16) T Xs[64 * XS];  // x of the chunk [t][p]
  __shared__ __align__(16) T Gs[64 * GS];  // causal Gamma [t][k]
  __shared__ __align__(16) T Ys[64 * XS];  // output rows [t][p]
  // per-token weight arrays [MP][WQ]: the row stride of 68 floats spreads the
  // stores of one wave (4 tokens x 16 modes, or 8 x 8) over distinct LDS banks
  constexpr int WQ = kQ + 4;
  __shared__ __align__(16) float W[8 * MP * WQ];
  float* P_O = W;                  // [MP][Q] c e^{-rA_t}        (Gamma rows)
  float* P_Vt = W + MP * WQ;       // [MP][Q] kappa e^{rA_t}, safe modes (Gamma columns)
  float* P_c = W + 2 * MP * WQ;    // [MP][Q] c, kappa (modes past the factorisation bound)
  float* P_k = W + 3 * MP * WQ;
  // chunk log-decays l_{t,m} [MP][Q], hi and lo parts, in two buffers: chunk c's in
  // buffer c & 1, formed while the previous chunk is processed
  float* P_L = W + 4 * MP * WQ;
  // the readout and update weights in the operand type, laid out for the operand reads:
  // Om [t][m] = c e^{-rA_t} E_m (four modes per read), Vm [m][t] = kappa e^{-r(A_Q-A_t)} upd
  // (eight tokens per read)
  constexpr int OS = MP + 4, VS = kBf16 ? kQ + 8 : kQ + 4;
  __shared__ __align__(16) T Om[kQ * OS];
  __shared__ __align__(16) T Vm[MP * VS];
  __shared__ __align__(16) float s_ren[MP];  // the state's rescale factor of the chunk (1: none)
  __shared__ float s_E2[2][MP];

  // Gamma tiles above the diagonal that the intra product reads are never written
  for (int i = tid; i < 64 * GS; i += NT) Gs[i] = (T)0.0f;
  if (tid < MP) s_E2[0][tid] = s_E2[1][tid] = 1.0f;
  // the mode of this thread's (token, mode) pairs: its rate and log time constant
  const int wm = tid % MP;
  const float wtau = (wm < M) ? p.tau[wm] : 1.0f;
  const float wr = (wm < M) ? 1.0f / wtau : 0.0f, wlnt = (wm < M) ? logf(wtau) : 0.0f;
  // without logits the scores of a token are -alpha ln tau_m, whose largest lies at the
  // smallest or the largest ln tau: the value the group reduction would find
  const float lnt_lo = group_allreduce<MP>(wm < M ? wlnt : INFINITY, [](float a, float b) { return fminf(a, b); });
  const float lnt_hi = group_allreduce<MP>(wm < M ? wlnt : -INFINITY, [](float a, float b) { return fmaxf(a, b); });
  // the rates of all modes for the log-decay sums (lane = token)
  __shared__ float s_rr[MP];
  if (tid < MP) s_rr[tid] = wr;
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
  const unsigned xs32 = (unsigned)(H * P);
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const int64_t lg_st = (int64_t)H * M;
  constexpr int E16 = 16 / (int)sizeof(T);  // elements per 16-byte vector
  constexpr int CPR = CW / E16;             // 16-byte vectors per row of this workgroup's columns
  constexpr int XV = 64 * CPR / NT;         // 16-byte vectors of x (and y) per thread and chunk
  static_assert(XV * NT == 64 * CPR, "the x tile splits evenly over the threads");

  // Per chunk c, three barriers:
  //   1. x(c) into LDS, the weights of c (from its log-decays), the loads of x(c + 1)
  //   2. the Gamma tiles of c; the log-decays of c + 1 (the other buffer); the loads of
  //      the controls of c + 2
  //   3. readout and state update of c
  //   4. the output rows of c to global memory (no barrier: the next chunk writes no
  //      array this phase reads)
  // x and the logits of a chunk are loaded one chunk ahead into registers, the
  // per-token controls (step, order, lambda) two chunks ahead.  Every global access
  // of the loop goes through a buffer resource whose range ends at the chunk's last
  // valid token, with per-lane offsets fixed for the whole sequence (past d_h, past
  // the modes: an offset beyond every range): out-of-range loads return zeros and
  // out-of-range stores are dropped, so the loop issues every access unconditionally
  // and a register filled by a load is never merged with a default value.
  constexpr unsigned kOut = 0x80000000u;
  const unsigned xs_b = xs32 * (unsigned)sizeof(T);  // bytes between consecutive tokens of x, y
  auto nv_of = [&](int c) { return max(0, min(kQ, L - c * kQ)); };
  auto span = [](int nv, int64_t stride, int64_t tail) {  // bytes of rows 0 .. nv - 1
    return nv > 0 ? (int)min(((int64_t)(nv - 1) * stride + tail), (int64_t)kOut - 1) : 0;
  };
  auto rsrc = [](const void* base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
  };
  unsigned xoff[XV];  // byte offsets of this thread's 16-byte vectors of the x / y tiles
#pragma unroll
  for (int j = 0; j < XV; ++j) {
    const int i = tid + NT * j, t = i / CPR, col = (i - t * CPR) * E16;
    xoff[j] = (p0 + col < P) ? (unsigned)t * xs_b + (unsigned)(col * (int)sizeof(T)) : kOut;
  }
  const int xtail = (P - p0) * (int)sizeof(T);
  int4 xr[XV];
  float dt_q = 0.0f, al_q = 1.0f, lam_q = 1.0f;  // raw controls of the chunk after the next one in flight
  constexpr int NPR = (kQ * MP + NT - 1) / NT;  // (token, mode) pairs per thread: pair = t MP + m = tid + NT j
  float rlr[NPR], wlr[NPR];           // the read / write logits of this thread's pairs
  unsigned loff[NPR];
#pragma unroll
  for (int j = 0; j < NPR; ++j) {
    const int pr = tid + NT * j, t = pr / MP;
    loff[j] = (pr < kQ * MP && wm < M) ? (unsigned)(t * (H * M) + wm) * 4u : kOut;
  }
  const bool own_wl = wl_bh && wl_bh != rl_bh;  // a separate write-logit array
  auto prefetch_x = [&](int c) {
    const int t0 = c * kQ, nv = nv_of(c);
    const auto rx = rsrc(xg + (int64_t)t0 * xstride, span(nv, xs_b, xtail));
#pragma unroll
    for (int j = 0; j < XV; ++j) xr[j] = __builtin_bit_cast(int4, __builtin_amdgcn_raw_buffer_load_b128(rx, xoff[j], 0, 0));
    const int lb = span(nv, (int64_t)H * M * 4, (int64_t)M * 4);
    const auto rr = rsrc(rl_bh ? rl_bh + (int64_t)t0 * lg_st : p.tau, rl_bh ? lb : 0);
    const auto rw = rsrc(own_wl ? wl_bh + (int64_t)t0 * lg_st : p.tau, own_wl ? lb : 0);
#pragma unroll
    for (int j = 0; j < NPR; ++j) {
      rlr[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, loff[j], 0, 0));
      wlr[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rw, loff[j], 0, 0));
    }
  };
  auto load_controls = [&](int c) {  // lane = token; zeros past the sequence
    const int t0 = c * kQ, nv = nv_of(c);
    const auto rd = rsrc(dt_bh + (int64_t)t0 * H, span(nv, (int64_t)H * 4, 4));
    const auto ra = rsrc(al_bh + (int64_t)t0 * p.as1, span(nv, (int64_t)p.as1 * 4, 4));
    const auto rl = rsrc(lm_bh ? lm_bh + (int64_t)t0 * p.ls1 : p.tau, lm_bh ? span(nv, (int64_t)p.ls1 * 4, 4) : 0);
    dt_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rd, (unsigned)(lane * H) * 4u, 0, 0));
    al_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ra, (unsigned)(lane * p.as1) * 4u, 0, 0));
    lam_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rl, (unsigned)(lane * p.ls1) * 4u, 0, 0));
  };
  // the effective step of this lane's token (0 past the sequence) from the raw controls
  auto eff_step = [&](int c) {
    const float s_eff = lm_bh ? step_factor(lam_q, al_q) : 1.0f;
    return (lane < nv_of(c)) ? dt_q * s_eff : 0.0f;
  };
  // the output rows of chunk c from LDS to global memory, 16 bytes per thread
  auto store_y = [&](int c) {
    const auto ry = rsrc(yg + (int64_t)c * kQ * xstride, span(nv_of(c), xs_b, xtail));
#pragma unroll
    for (int j = 0; j < XV; ++j) {
      const int i = tid + NT * j, t = i / CPR, col = (i - t * CPR) * E16;
      const int4 v = *reinterpret_cast<const int4*>(Ys + t * XS + col);
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4_t, v), ry, xoff[j], 0, 0);
    }
  };
  // the state entering chunk c as stored for the backward (modes past M, columns past
  // d_h and the second token half store nothing)
  unsigned ckoff[MB * 4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = mb * 16 + lg * 4 + r;
      ckoff[mb * 4 + r] = (active && half == 0 && m < M && pc < P) ? (unsigned)(m * P + pc) * 4u : kOut;
    }
  float dtt_c, al_c;  // the effective step and order of the current chunk (lane = token)
  load_controls(0);
  dtt_c = eff_step(0);
  al_c = al_q;
  load_controls(1);
  prefetch_x(0);
  barrier();  // the rates and scales in LDS
  chunk_log_decays<MP, NW>(dtt_c, s_rr, P_L, P_L + MP * WQ);
  barrier();  // the log-decays of the first chunk in LDS

  for (int c = 0; c < nchunks; ++c) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    const float* Ecur = s_E2[c & 1];
    float* Enext = s_E2[(c + 1) & 1];
    const float* P_lh = P_L + (c & 1) * 2 * MP * WQ;
    const float* P_ll = P_lh + MP * WQ;
    // ---- x of the chunk into LDS (zeros past the sequence and past d_h)
#pragma unroll
    for (int j = 0; j < XV; ++j) {
      const int i = tid + NT * j, t = i / CPR, col = (i - t * CPR) * E16;
      *reinterpret_cast<int4*>(Xs + t * XS + col) = xr[j];
    }
    if (CKPT || ckpt) {  // the state entering this chunk
      const auto rk = rsrc(ckpt + ((int64_t)bh * (nchunks + 1) + c) * M * P, M * P * 4);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mb * 16 + lg * 4 + r;
          const float v = S[mb][r] * Ecur[m < MP ? m : 0];
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), rk, ckoff[mb * 4 + r], 0, 0);
        }
    }
    const bool over = lane < MP && lane < M && !(P_lh[(lane < MP ? lane : 0) * WQ + kQ - 1] <= kNfSafe);
    const int unsafe = (int)(__ballot(over) & ((MP >= 32) ? 0xffffffffull : ((1ull << MP) - 1)));
    // ---- per (token, mode) weights: pair = t MP + m, m = wm
#pragma unroll
    for (int j = 0; j < NPR; ++j) {
      const int pr = tid + NT * j, t = pr / MP, m = wm;
      if (pr >= kQ * MP) break;  // wave-uniform
      const float dtt = __shfl(dtt_c, t, 64), al = __shfl(al_c, t, 64);
      const bool valid = t < nv;
      const float prior = -al * wlnt;
      const float zc = (m < M) ? prior + rlr[j] : -INFINITY;
      const float zw = (m < M) ? prior + wlr[j] : -INFINITY;
      const float lhQ = P_lh[m * WQ + kQ - 1], llQ = P_ll[m * WQ + kQ - 1];
      const float Enew = Ecur[m] * fexp(-lhQ);
      const bool ren = !(Enew >= kNfFloor);
      const float upd = ren ? 1.0f : fast_rcp(Enew);
      const float lh = P_lh[m * WQ + t], ll = P_ll[m * WQ + t];
      const float dQ = __expf(-fmaxf(ell_diff(lhQ, llQ, lh, ll), 0.0f));  // e^{-(l_Q - l_t)}
      if constexpr (CKPT) {  // the state update only: the write weights
        const float ww = valid ? group_softmax<MP>((rl_bh == wl_bh) ? zc : zw) : 0.0f;
        const float kap = one_minus_exp_neg(dtt * wr) * ww;
        Vm[m * VS + t] = (T)(kap * dQ * upd);
      } else {
        float cw;
        if (!rl_bh) {  // the scores are the priors: their maximum is known
          const float e = __expf(zc - fmaxf(-al * lnt_lo, -al * lnt_hi));
          const float sum = group_allreduce<MP>(e, [](float a, float b) { return a + b; });
          cw = valid ? e * fast_rcp(sum) : 0.0f;
        } else {
          cw = valid ? group_softmax<MP>(zc) : 0.0f;
        }
        const float ww = (rl_bh == wl_bh) ? cw : (valid ? group_softmax<MP>(zw) : 0.0f);
        const bool safe = lhQ <= kNfSafe;
        const float kap = one_minus_exp_neg(dtt * wr) * ww;
        const float om = cw * fexp(-lh);
        P_O[m * WQ + t] = om;
        P_Vt[m * WQ + t] = safe ? kap * fexp(lh) : 0.0f;
        Om[t * OS + m] = (T)(om * Ecur[m]);
        Vm[m * VS + t] = (T)(kap * dQ * upd);
        if (unsafe) {  // wave-uniform
          P_c[m * WQ + t] = cw;
          P_k[m * WQ + t] = kap;
        }
      }
      if (pr < MP) {
        Enext[m] = ren ? 1.0f : Enew;
        s_ren[m] = ren ? Enew : 1.0f;
      }
    }
    prefetch_x(c + 1);  // this chunk's x and logits are consumed (past the end: nothing is read)
    barrier();  // x and the weights in LDS

    if constexpr (!CKPT) {
    // ---- causal Gamma tiles [t][k] (float32 matrix cores, modes as K)
    for (int tile = wave; tile < 10; tile += NW) {
      const int tb = tile_row(tile), kb = tile_col(tile);
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
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
            if (t >= k) Gm[r] += P_c[m * WQ + t] * P_k[m * WQ + k] * ell_decay(P_lh + m * WQ, P_ll + m * WQ, t, k);
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
        Gs[t * GS + k] = (T)keep_if_ge(Gm[r], t, k);
      }
    }
    }  // !CKPT
    // ---- the next chunk's per-token controls and log-decays (the other buffer)
    if (c + 1 < nchunks) {
      dtt_c = eff_step(c + 1);
      al_c = al_q;
      float* N_lh = P_L + ((c + 1) & 1) * 2 * MP * WQ;
      chunk_log_decays<MP, NW>(dtt_c, s_rr, N_lh, N_lh + MP * WQ);
    }
    load_controls(c + 2);
    barrier();  // Gamma and the next log-decays in LDS

    if (active) {
      if constexpr (!CKPT) {
      // ---- readout, intra-chunk product and skip term, row blocks of 16 tokens
      Frag<T> Sf;  // the state as a B operand: slot s < 4 mode 4 lg + s, s >= 4 mode 16 + 4 lg + s - 4
#pragma unroll
      for (int s = 0; s < 4; ++s) frag_set(Sf, s, S[0][s]);
#pragma unroll
      for (int s = 0; s < 4; ++s) frag_set(Sf, 4 + s, MB > 1 ? S[MB - 1][s] : 0.0f);
#pragma unroll
      for (int tq = 0; tq < 4 / NH; ++tq) {
        const int tb = half * (4 / NH) + tq;  // row block of 16 tokens
        const int t = tb * 16 + li;            // this lane's token (Gamma and O row)
        // the transposed products (operands swapped): lane (li, lg) accumulates the
        // outputs of token t at columns cg 16 + 4 lg .. + 3, stored as one vector
        floatx4 Y = {0.f, 0.f, 0.f, 0.f};
        // slots as in Sf; modes past MP (lane groups beyond MP / 4) are zero
        const Frag<T> Of = (lg * 4 < MP) ? frag_load4x2(Om + t * OS + lg * 4, Om + t * OS + 16 + lg * 4, MB > 1)
                                         : frag_zero<T>();
        mma(Y, Sf, Of);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          if (kk > tb / 2) break;  // wave-uniform
          const Frag<T> a = frag_load8(Gs + t * GS + kk * 32 + lg * 8);
          const Frag<T> bx = frag_load_rows(Xs, XS, kk * 32 + lg * 8, cg * 16);
          mma(Y, bx, a);
        }
        float xv[4];
        load4(Xs + t * XS + cg * 16 + lg * 4, xv);
#pragma unroll
        for (int r = 0; r < 4; ++r) Y[r] += Dh * xv[r];
        store4(Ys + t * XS + cg * 16 + lg * 4, Y);
      }
      }  // !CKPT

      // ---- state update S_m <- (rescale) S_m + V^T x, V = kappa e^{-r(A_Q - A_k)} upd
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mb * 16 + lg * 4 + r;
          if (m < MP) S[mb][r] *= s_ren[m];
        }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const Frag<T> bx = frag_load_rows(Xs, XS, kt * 32 + lg * 8, cg * 16);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int m = mb * 16 + li;  // A-operand row (mode)
          const Frag<T> Vf = (m < MP) ? frag_load8(Vm + m * VS + kt * 32 + lg * 8) : frag_zero<T>();
          mma(S[mb], Vf, bx);
        }
      }
    }
    barrier();  // output rows in LDS; every array of this chunk is consumed
    if constexpr (!CKPT) store_y(c);
  }

  float* fin_ck = ckpt ? ckpt + ((int64_t)bh * (nchunks + 1) + nchunks) * M * P : nullptr;
  float* fin = (!CKPT && p.final_state) ? p.final_state + sbase : nullptr;
  if ((fin || fin_ck) && active && half == 0) {
    const float* Ef = s_E2[nchunks & 1];  // written before the last chunk's weights barrier
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb * 16 + lg * 4 + r;
        if (m < M && pc < P) {
          const float v = S[mb][r] * Ef[m];
          if (fin) fin[(int64_t)m * P + pc] = v;
          if (fin_ck) fin_ck[(int64_t)m * P + pc] = v;
        }
      }
  }
}

// ------------------------------------------------ forward, split waves
//
// Head dims above 128 with up to 16 modes: one workgroup of 16 waves per (batch,
// head, 128 columns), in two roles with one barrier per iteration.  Producer waves
// 8 .. 15 form, in iteration i, the weights of chunk i + 1 (from the log-decays
// formed one iteration earlier) and the Gamma tiles of chunk i (from the weights
// formed one iteration earlier).  Consumer waves 0 .. 7 form the log-decays of
// chunk i + 2 (two modes each), and each owns 16 columns where, in iteration i, it
// runs chunk i - 1: x into its own columns of LDS, readout, intra-chunk product and
// skip term (outputs stored from registers), the state update.  The per-chunk work
// that does not depend on the state thus overlaps the recurrence; buffers are kept
// for as many chunks as are in flight (log-decays, readout and update weights:
// three; Gamma and its factors: two).
// KEEP: ckpt receives the state entering every chunk and the final state (the
// caller's kept chunk states); without it ckpt is not read.
template <typename T, int MP, bool KEEP>
__global__ void __launch_bounds__(1024) frac_nfree_fwd_split_kernel(ScanParams p, float* __restrict__ ckpt_arg) {
  float* const ckpt = KEEP ? ckpt_arg : nullptr;
  constexpr bool kBf16 = sizeof(T) == 2;
  constexpr int MB = (MP + 15) / 16;
  constexpr int CW = 128, NPW = 8, NPT = 64 * NPW;  // columns, producer waves, producer threads
  constexpr int XS = kBf16 ? CW + 8 : CW + 4;
  constexpr int GS = kBf16 ? 64 + 8 : 64 + 4;
  constexpr int WQ = kQ + 4;
  constexpr int OS = MP + 4, VS = kBf16 ? kQ + 8 : kQ + 4;
  constexpr int ES = (int)sizeof(T);
  static_assert(NPT % MP == 0, "every (token, mode) pair of a producer thread has the same mode");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const bool producer = wave >= 8;
  const int pt = tid - NPT, pw = wave - 8;  // producer thread and wave (when producer)
  const int L = p.L, H = p.H, P = p.P, M = p.M;
  const int nps = (P + CW - 1) / CW;
  const int ps = blockIdx.x % nps, bh = blockIdx.x / nps, b = bh / H, h = bh - b * H;
  const int p0 = ps * CW;
  const int cg = wave & 7, pc = p0 + cg * 16 + li;  // consumer column group and lane column
  const bool active = !producer && p0 + cg * 16 < P;
  const int nchunks = (L + kQ - 1) / kQ;

  __shared__ __align__(16) T Xs[64 * XS];          // x of the consumers' chunk [t][p]
  __shared__ __align__(16) T Gb[2][64 * GS];       // Gamma [t][k] of chunk j in Gb[j & 1]
  __shared__ __align__(16) float LDb[3][2 * MP * WQ];  // log-decays (hi, lo) [MP][Q] of chunk j in LDb[j % 3]
  __shared__ __align__(16) float Wb[2][4 * MP * WQ];   // Gamma factors c e^{-l}, kappa e^{l}; c, kappa (unsafe modes)
  __shared__ __align__(16) T Omb[3][kQ * OS];      // readout weights [t][m] of chunk j in slot j % 3
  __shared__ __align__(16) T Vmb[3][MP * VS];      // update weights [m][t]
  __shared__ __align__(16) float s_ren[3][MP];     // the state's rescale factor of chunk j
  __shared__ float s_Ein[3][MP];                   // the state scale entering chunk j
  __shared__ float s_E[2][MP];                     // the running state scale (producers)
  __shared__ float s_rr[MP];
  __shared__ float s_dtt[3][kQ], s_al[3][kQ];      // effective step and order of chunk j's tokens in slot j % 3

  for (int i = tid; i < 2 * 64 * GS; i += 1024) (&Gb[0][0])[i] = (T)0.0f;  // tiles above the diagonal stay zero
  const int wm = (producer ? pt : tid) % MP;
  const float wtau = (wm < M) ? p.tau[wm] : 1.0f;
  const float wr = (wm < M) ? 1.0f / wtau : 0.0f, wlnt = (wm < M) ? logf(wtau) : 0.0f;
  const float lnt_lo = group_allreduce<MP>(wm < M ? wlnt : INFINITY, [](float a, float b) { return fminf(a, b); });
  const float lnt_hi = group_allreduce<MP>(wm < M ? wlnt : -INFINITY, [](float a, float b) { return fmaxf(a, b); });
  if (tid < MP) {
    s_rr[tid] = wr;
    s_E[0][tid] = 1.0f;
  }

  constexpr unsigned kOut = 0x80000000u;
  const int64_t xstride = (int64_t)H * P;
  const unsigned xs_b = (unsigned)(H * P) * (unsigned)ES;
  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * P + p0;
  T* yg = reinterpret_cast<T*>(p.y) + (((int64_t)b * L) * H + h) * P + p0;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const bool own_wl = wl_bh && wl_bh != rl_bh;
  const int64_t lg_st = (int64_t)H * M;
  const int xtail = (P - p0) * ES;
  auto nv_of = [&](int c) { return (c >= 0 && c < nchunks) ? min(kQ, L - c * kQ) : 0; };
  auto span = [](int nv, int64_t stride, int64_t tail) {
    return nv > 0 ? (int)min(((int64_t)(nv - 1) * stride + tail), (int64_t)kOut - 1) : 0;
  };
  auto rsrc = [](const void* base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
  };

  // ---- producer state: raw controls two chunks ahead (lane = token), the effective
  // step and order of the chunk whose weights come next, the logits of those weights
  constexpr int NPR = (kQ * MP + NPT - 1) / NPT;
  float dt_q = 0.0f, al_q = 1.0f, lam_q = 1.0f;  // raw controls of a chunk two ahead (consumers, lane = token)
  float rlr[NPR] = {}, wlr[NPR] = {};
  unsigned loff[NPR];
#pragma unroll
  for (int j = 0; j < NPR; ++j) {
    const int pr = pt + NPT * j, t = pr / MP;
    loff[j] = (producer && pr < kQ * MP && wm < M) ? (unsigned)(t * (H * M) + wm) * 4u : kOut;
  }
  auto load_controls = [&](int c) {
    const int t0 = c * kQ, nv = nv_of(c);
    const auto rd = rsrc(dt_bh + (int64_t)t0 * H, span(nv, (int64_t)H * 4, 4));
    const auto ra = rsrc(al_bh + (int64_t)t0 * p.as1, span(nv, (int64_t)p.as1 * 4, 4));
    dt_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rd, (unsigned)(lane * H) * 4u, 0, 0));
    al_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ra, (unsigned)(lane * p.as1) * 4u, 0, 0));
    if (lm_bh) {  // read only where lambda is given (the value is used only then)
      const auto rl = rsrc(lm_bh + (int64_t)t0 * p.ls1, span(nv, (int64_t)p.ls1 * 4, 4));
      lam_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rl, (unsigned)(lane * p.ls1) * 4u, 0, 0));
    }
  };
  auto eff_step = [&](int c) {
    const float s_eff = lm_bh ? step_factor(lam_q, al_q) : 1.0f;
    return (lane < nv_of(c)) ? dt_q * s_eff : 0.0f;
  };
  auto load_logits = [&](int c) {  // read only where given (the values are used only then)
    const int t0 = c * kQ, nv = nv_of(c);
    const int lb = span(nv, (int64_t)H * M * 4, (int64_t)M * 4);
    if (rl_bh) {
      const auto rr = rsrc(rl_bh + (int64_t)t0 * lg_st, lb);
#pragma unroll
      for (int j = 0; j < NPR; ++j) rlr[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, loff[j], 0, 0));
    }
    if (own_wl) {
      const auto rw = rsrc(wl_bh + (int64_t)t0 * lg_st, lb);
#pragma unroll
      for (int j = 0; j < NPR; ++j) wlr[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rw, loff[j], 0, 0));
    }
  };
  // the per-mode log-decays of chunk c from this lane's effective step (wave wi of
  // eight: modes wi, wi + 8, ..), and the token's step and order for the weights
  auto log_decays = [&](int c, float dtt, float al, int wi) {
    float* lh = LDb[c % 3];
    if (wi == 0) {
      s_dtt[c % 3][lane] = dtt;
      s_al[c % 3][lane] = al;
    }
#pragma unroll
    for (int m0 = 0; m0 < MP; m0 += NPW) {
      const int m = m0 + wi;
      if (m0 + NPW > MP && m >= MP) break;  // wave-uniform
      const double v = wave_inclusive_sum_f64((double)capped_exponent(s_rr[m], dtt));
      const float hi = (float)v;
      lh[m * WQ + lane] = hi;
      lh[MP * WQ + m * WQ + lane] = (float)(v - (double)hi);
    }
  };
  auto unsafe_of = [&](int c) {
    const float* lh = LDb[c % 3];
    const bool over = lane < MP && lane < M && !(lh[(lane < MP ? lane : 0) * WQ + kQ - 1] <= kNfSafe);
    return (int)(__ballot(over) & ((MP >= 32) ? 0xffffffffull : ((1ull << MP) - 1)));
  };
  // the weights of chunk c: the Gamma factors, the readout and update weights, the
  // state scale and rescale
  auto weights = [&](int c) {
    const float* P_lh = LDb[c % 3];
    const float* P_ll = P_lh + MP * WQ;
    float* W = Wb[c & 1];
    T* Om = Omb[c % 3];
    T* Vm = Vmb[c % 3];
    const float* Ecur = s_E[c & 1];
    float* Enext = s_E[(c + 1) & 1];
    const int nv = nv_of(c), unsafe = unsafe_of(c);
#pragma unroll
    for (int j = 0; j < NPR; ++j) {
      const int pr = pt + NPT * j, t = pr / MP, m = wm;
      if (pr >= kQ * MP) break;  // wave-uniform
      const float dtt = s_dtt[c % 3][t], al = s_al[c % 3][t];
      const bool valid = t < nv;
      const float prior = -al * wlnt;
      const float zc = (m < M) ? prior + (rl_bh ? rlr[j] : 0.0f) : -INFINITY;
      const float zw = (m < M) ? prior + (own_wl ? wlr[j] : 0.0f) : -INFINITY;
      const float lhQ = P_lh[m * WQ + kQ - 1], llQ = P_ll[m * WQ + kQ - 1];
      const float Ec = Ecur[m];
      const float Enew = Ec * fexp(-lhQ);
      const bool ren = !(Enew >= kNfFloor);
      const float upd = ren ? 1.0f : fast_rcp(Enew);
      const float lh = P_lh[m * WQ + t], ll = P_ll[m * WQ + t];
      const float dQ = __expf(-fmaxf(ell_diff(lhQ, llQ, lh, ll), 0.0f));  // e^{-(l_Q - l_t)}
      float cw;
      if (!rl_bh) {  // the scores are the priors: their maximum is known
        const float e = __expf(zc - fmaxf(-al * lnt_lo, -al * lnt_hi));
        const float sum = group_allreduce<MP>(e, [](float a, float b) { return a + b; });
        cw = valid ? e * fast_rcp(sum) : 0.0f;
      } else {
        cw = valid ? group_softmax<MP>(zc) : 0.0f;
      }
      const float ww = (rl_bh == wl_bh) ? cw : (valid ? group_softmax<MP>(zw) : 0.0f);
      const bool safe = lhQ <= kNfSafe;
      const float kap = one_minus_exp_neg(dtt * wr) * ww;
      const float om = cw * fexp(-lh);
      W[m * WQ + t] = om;
      W[MP * WQ + m * WQ + t] = safe ? kap * fexp(lh) : 0.0f;
      Om[t * OS + m] = (T)(om * Ec);
      Vm[m * VS + t] = (T)(kap * dQ * upd);
      if (unsafe) {  // wave-uniform
        W[2 * MP * WQ + m * WQ + t] = cw;
        W[3 * MP * WQ + m * WQ + t] = kap;
      }
      if (pr < MP) {
        Enext[m] = ren ? 1.0f : Enew;
        s_ren[c % 3][m] = ren ? Enew : 1.0f;
        s_Ein[c % 3][m] = Ec;
      }
    }
  };
  // causal Gamma tile `tile` of chunk c (modes as K; one exponential per pair for the
  // modes past the factorisation bound)
  auto gamma = [&](int c, int tile) {
    const float* P_lh = LDb[c % 3];
    const float* P_ll = P_lh + MP * WQ;
    const float* W = Wb[c & 1];
    T* Gs = Gb[c & 1];
    const int unsafe = unsafe_of(c);
    {
      const int tb = tile_row(tile), kb = tile_col(tile);
      floatx4 Gm = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < (MP + 3) / 4; ++q) {
        const int m = q * 4 + lg;
        const float av = (m < MP) ? W[m * WQ + tb * 16 + li] : 0.0f;
        const float bv = (m < MP) ? W[MP * WQ + m * WQ + kb * 16 + li] : 0.0f;
        Gm = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, Gm, 0, 0, 0);
      }
      if (unsafe) {
        for (int m = 0; m < MP; ++m) {
          if (!((unsafe >> m) & 1)) continue;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
            if (t >= k)
              Gm[r] += W[2 * MP * WQ + m * WQ + t] * W[3 * MP * WQ + m * WQ + k] * ell_decay(P_lh + m * WQ, P_ll + m * WQ, t, k);
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
        Gs[t * GS + k] = (T)keep_if_ge(Gm[r], t, k);
      }
    }
  };

  // ---- consumer state: the state slice, x of the next chunk (lane = token, two
  // 16-byte vectors of this wave's 16 columns)
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
  constexpr int XV = 16 * ES / 16;  // 16-byte vectors per row of a wave's 16 columns
  int4 xr[XV];
  unsigned xoff[XV];
#pragma unroll
  for (int v = 0; v < XV; ++v) {
    const int col = cg * 16 + v * (16 / ES);
    xoff[v] = (active && p0 + col < P) ? (unsigned)lane * xs_b + (unsigned)(col * ES) : kOut;
  }
  auto load_x = [&](int c) {
    const auto rx = rsrc(xg + (int64_t)max(c, 0) * kQ * xstride, span(nv_of(c), xs_b, xtail));
#pragma unroll
    for (int v = 0; v < XV; ++v) xr[v] = __builtin_bit_cast(int4, __builtin_amdgcn_raw_buffer_load_b128(rx, xoff[v], 0, 0));
  };
  unsigned ckoff[MB * 4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = mb * 16 + lg * 4 + r;
      ckoff[mb * 4 + r] = (active && m < M && pc < P) ? (unsigned)(m * P + pc) * 4u : kOut;
    }
  // the state scaled by E, as the state entering chunk c (slot c of the kept states)
  auto store_state = [&](int c, const float* E) {
    const auto rk = rsrc(ckpt + ((int64_t)bh * (nchunks + 1) + c) * M * P, M * P * 4);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb * 16 + lg * 4 + r;
        const float v = S[mb][r] * E[m < MP ? m : 0];
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), rk, ckoff[mb * 4 + r], 0, 0);
      }
  };
  // the outputs of a row block: lane (li, lg) holds token 16 tb + li, columns cg 16 + 4 lg .. + 3
  unsigned yoff[4];
#pragma unroll
  for (int tb = 0; tb < 4; ++tb) {
    const int col = cg * 16 + lg * 4;
    yoff[tb] = (active && p0 + col < P) ? (unsigned)(tb * 16 + li) * xs_b + (unsigned)(col * ES) : kOut;
  }

  // ---- prologue: the log-decays of chunks 0 and 1 (consumers), then the weights of chunk 0
  if (producer) {
    load_logits(0);
  } else {
    load_x(0);
    load_controls(0);
  }
  __syncthreads();  // the rates and scales in LDS
  if (!producer) {
    log_decays(0, eff_step(0), al_q, cg);
    load_controls(1);
    log_decays(1, eff_step(1), al_q, cg);
    load_controls(2);
  }
  __syncthreads();  // the first log-decays in LDS
  if (producer) {
    weights(0);
    load_logits(1);
  }
  __syncthreads();  // the weights of chunk 0 in LDS
  if constexpr (KEEP) {
    if (!producer) store_state(0, s_Ein[0]);  // the initial state (scale 1)
  }

  for (int it = 0; it <= nchunks; ++it) {
    if (producer) {
      if (it + 1 < nchunks) weights(it + 1);
      if (it < nchunks)
        for (int tile = pw; tile < 10; tile += NPW) gamma(it, tile);
      load_logits(it + 2);
    } else {
      // log-decays of chunk it + 2 from the controls loaded one iteration ago
      if (it + 2 < nchunks) log_decays(it + 2, eff_step(it + 2), al_q, cg);
      load_controls(it + 3);
      if (it >= 1) {
      const int c = it - 1, slot = c % 3;
      const int nv = nv_of(c);
      const T* Gs = Gb[c & 1];
      const T* Om = Omb[slot];
      const T* Vm = Vmb[slot];
      // x of the chunk into this wave's columns of LDS (lane = token)
#pragma unroll
      for (int v = 0; v < XV; ++v) *reinterpret_cast<int4*>(Xs + lane * XS + cg * 16 + v * (16 / ES)) = xr[v];
      load_x(c + 1);
      Frag<T> Sf;  // the state as a B operand: slot s < 4 mode 4 lg + s, s >= 4 mode 16 + 4 lg + s - 4
#pragma unroll
      for (int s = 0; s < 4; ++s) frag_set(Sf, s, S[0][s]);
#pragma unroll
      for (int s = 0; s < 4; ++s) frag_set(Sf, 4 + s, MB > 1 ? S[MB - 1][s] : 0.0f);
      const auto ry = rsrc(yg + (int64_t)c * kQ * xstride, span(nv, xs_b, xtail));
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        const int t = tb * 16 + li;
        floatx4 Y = {0.f, 0.f, 0.f, 0.f};  // transposed products: token t, columns cg 16 + 4 lg .. + 3
        const Frag<T> Of = (lg * 4 < MP) ? frag_load4x2(Om + t * OS + lg * 4, Om + t * OS + 16 + lg * 4, MB > 1)
                                         : frag_zero<T>();
        mma(Y, Sf, Of);
#pragma unroll
        for (int kk = 0; kk <= tb / 2; ++kk)
          mma(Y, frag_load_rows(Xs, XS, kk * 32 + lg * 8, cg * 16), frag_load8(Gs + t * GS + kk * 32 + lg * 8));
        float xv[4];
        load4(Xs + t * XS + cg * 16 + lg * 4, xv);
#pragma unroll
        for (int r = 0; r < 4; ++r) Y[r] += Dh * xv[r];
        if constexpr (kBf16) {
          const bf16x4 o = bf16x4{(bf16)Y[0], (bf16)Y[1], (bf16)Y[2], (bf16)Y[3]};
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, o), ry, yoff[tb], 0, 0);
        } else {
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4_t, Y), ry, yoff[tb], 0, 0);
        }
      }
      // ---- state update S_m <- (rescale) S_m + V^T x
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mb * 16 + lg * 4 + r;
          if (m < MP) S[mb][r] *= s_ren[slot][m];
        }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const Frag<T> bx = frag_load_rows(Xs, XS, kt * 32 + lg * 8, cg * 16);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int m = mb * 16 + li;
          const Frag<T> Vf = (m < MP) ? frag_load8(Vm + m * VS + kt * 32 + lg * 8) : frag_zero<T>();
          mma(S[mb], Vf, bx);
        }
      }
      // the state entering the next chunk, stored at the end of this one (a wait for
      // the loads issued at its start would also wait for these stores)
      if constexpr (KEEP) {
        if (c + 1 < nchunks) store_state(c + 1, s_Ein[(c + 1) % 3]);
      }
      }  // it >= 1
    }
    __syncthreads();  // this iteration's log-decays, weights and Gamma in LDS
  }

  float* fin_ck = ckpt ? ckpt + ((int64_t)bh * (nchunks + 1) + nchunks) * M * P : nullptr;
  float* fin = p.final_state ? p.final_state + sbase : nullptr;
  if ((fin || fin_ck) && active) {
    const float* Ef = s_E[nchunks & 1];  // the scale after the last chunk (written by its weights)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb * 16 + lg * 4 + r;
        if (m < M && pc < P) {
          const float v = S[mb][r] * Ef[m];
          if (fin) fin[(int64_t)m * P + pc] = v;
          if (fin_ck) fin_ck[(int64_t)m * P + pc] = v;
        }
      }
  }
}

// ---------------------------------------------------------------- backward
//
// Reverse sweep over the chunks with the adjoint G_m (M x d_h per head, this
// workgroup's 128 or 64 columns) in accumulator registers and each chunk's entering
// state S0 read from the chunk states (the caller's forward kept them, or the
// checkpoint pass wrote them).  Per chunk, with H = dY X^T over this
// workgroup's columns (a partial sum over d_h) and l the chunk log-decays:
//   dx_t = sum_m kappa_{t,m} e^{-(l_Q - l_t)} G_m + sum_{t'>=t} Gamma_{t',t} dy_t' + D dy_t
//   dc_{t,m} = e^{-l_t} (S0_m . dy_t) + sum_{k<=t} H_{t,k} kappa_{k,m} e^{-(l_t - l_k)}
//   dk_{k,m} = e^{-(l_Q - l_k)} (G_m . x_k) + sum_{t>=k} H_{t,k} c_{t,m} e^{-(l_t - l_k)}
//   G_m <- e^{-l_Q} G_m + sum_t c_{t,m} e^{-l_t} dy_t
// dc and dk (the gradients of the read weight and of the write gain, partial over
// this workgroup's columns) go to the shared finishing kernels (frac_grads.hip),
// which form ddt, dalpha, dlambda and the logit gradients.

struct NfWork {
  const float* ckpt;  // [B H][nchunks + 1][M][P] states entering each chunk, then the final state
  float* F;           // [nps][B H][M] <dS_final, S_final>_m over this workgroup's columns
  float* I;           // [nps][B H][M] <S_init, dS_init>_m over this workgroup's columns
  float* dDp;         // [nps][B H] sum dy . x over this workgroup's columns
  float* dcp;         // [nps][B H L][M] <h_{t,m}, dy_t>: gradient of the read weight c_{t,m}
  float* dkp;         // [nps][B H L][M] <G_{t,m}, x_t>: gradient of the injection kappa_{t,m},
                      // the part through the adjoint carried in from the later chunks
  float* dkip;        // [nps][B H L][M] its part through the chunk's own readouts
};

// NW waves per workgroup over 16 NW columns of d_h, as the forward.  With 8 waves
// the per-token products and partials of row block tb are split: waves tb form
// S0 . dy and dc, waves 4 + tb form G . x, dk and the intra dk.
template <typename T, int MP, int NW = 4>
__global__ void __launch_bounds__(64 * NW, NW == 4 ? 2 : 1) frac_nfree_bwd_kernel(ScanParams p, NfWork wk) {
  constexpr bool kBf16 = sizeof(T) == 2;
  constexpr int MB = (MP + 15) / 16;
  constexpr int NT = 64 * NW, CW = 16 * NW;    // threads, columns of d_h per workgroup
  constexpr int XS = kBf16 ? CW + 8 : CW + 4;  // [t][p] tile stride
  constexpr int GS = kBf16 ? 64 + 8 : 64 + 4;  // [t][t'] tile stride
  constexpr int GQ = kBf16 ? CW + 8 : CW + 4;  // row stride of the adjoint [m][p]
  constexpr int KP = CW / 32;                  // 32-column K steps over this workgroup's columns
  constexpr bool kSplit = NW == 8;
  constexpr int WQ = kWQ;
  constexpr int NWA = 8;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int L = p.L, H = p.H, P = p.P, M = p.M;
  const int nps = (P + CW - 1) / CW;
  const int ps = blockIdx.x % nps, bh = blockIdx.x / nps, b = bh / H, h = bh - b * H;
  const int p0 = ps * CW, pc = p0 + wave * 16 + li;
  const bool active = p0 + wave * 16 < P;
  const int nchunks = (L + kQ - 1) / kQ;
  const bool doU = !kSplit || wave < 4, doZ = !kSplit || wave >= 4;  // this wave's per-token products

  __shared__ __align__(16) T Xs[64 * XS];                      // x [t][p]
  __shared__ __align__(16) T Ys[64 * XS];                      // dy [t][p]
  __shared__ __align__(16) T GT[64 * GS];                      // Gamma^T [t][t'], t' >= t
  constexpr int HS = 64 + 4;
  __shared__ __align__(16) float HT[64 * HS];                  // dY X^T [t][k], k <= t (float32)
  __shared__ __align__(16) T DX[kBf16 ? 64 * XS : 8];         // dx rows [t][p] (bfloat16 staging)
  // the adjoint [m][p] in the operand type: for bfloat16 a rounded value (GtH) and its
  // rounded remainder (GtL), formed once by the wave that owns the columns
  __shared__ __align__(16) T GtH[MP * GQ];
  __shared__ __align__(16) T GtL[kBf16 ? MP * GQ : 8];
  // the state entering the chunk [m][p], likewise (loaded by all threads, four columns each)
  __shared__ __align__(16) T S0H[MP * GQ];
  __shared__ __align__(16) T S0L[kBf16 ? MP * GQ : 8];
  __shared__ __align__(16) float W[NWA * MP * WQ];
  __shared__ float s_rr[MP], s_lnt[MP];
  __shared__ float red[NW][MP > 64 ? MP : 64];
  __shared__ float redD[NT];
  // a sum of the waves' partials, in wave order
  auto red_sum = [&](int m) {
    float v = red[0][m];
#pragma unroll
    for (int w = 1; w < NW; ++w) v += red[w][m];
    return v;
  };
  constexpr int SW = MP * WQ;
  float* P_O = W;             // c e^{-l}
  float* P_Vt = W + 1 * SW;   // kappa e^{l} (safe modes), kappa (modes past the factorisation bound)
  float* P_vq = W + 2 * SW;   // kappa e^{-(l_Q - l)}
  float* P_c = W + 3 * SW;    // c (modes past the factorisation bound)
  // chunk log-decays [MP][Q], hi and lo parts, in two buffers: chunk c's in buffer
  // c & 1, formed while the chunk after it is processed
  float* P_L = W + 4 * SW;

  for (int i = tid; i < 64 * GS; i += NT) GT[i] = (T)0.0f;
  for (int i = tid; i < 64 * HS; i += NT) HT[i] = 0.0f;
  if (tid < MP) {
    const float tau = (tid < M) ? p.tau[tid] : 1.0f;
    s_rr[tid] = (tid < M) ? 1.0f / tau : 0.0f;
    s_lnt[tid] = (tid < M) ? logf(tau) : 0.0f;
  }
  __syncthreads();

  // the adjoint of the final state and the final-state term <dS_final, S_final> per mode
  const int64_t sbase = (int64_t)bh * M * P;
  const float* ck_bh = wk.ckpt + (int64_t)bh * (nchunks + 1) * M * P;
  floatx4 G[MB];
  float fpart[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = mb * 16 + lg * 4 + r;
      float g = 0.0f;
      fpart[mb][r] = 0.0f;
      if (p.d_final_state && active && m < M && pc < P) {
        g = p.d_final_state[sbase + (int64_t)m * P + pc];
        fpart[mb][r] = g * ck_bh[(int64_t)nchunks * M * P + (int64_t)m * P + pc];
      }
      G[mb][r] = g;
    }
  // summed over the 16 columns of each lane group, then over the waves in order
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float v = group_allreduce<16>(fpart[mb][r], [](float x, float y) { return x + y; });
      const int m = mb * 16 + lg * 4 + r;
      if (li == 0 && m < MP) red[wave][m] = v;
    }
  __syncthreads();
  if (tid < MP && tid < M) wk.F[((int64_t)ps * p.Bsz * H + bh) * M + tid] = red_sum(tid);
  const float Dh = p.D ? p.D[h] : 0.0f;
  float dd_acc = 0.0f;

  const T* xg = reinterpret_cast<const T*>(p.x) + (((int64_t)b * L) * H + h) * P + p0;
  const T* yg = reinterpret_cast<const T*>(p.dy) + (((int64_t)b * L) * H + h) * P + p0;
  T* dxg = reinterpret_cast<T*>(p.dx) + (((int64_t)b * L) * H + h) * P + p0;
  const int64_t xstride = (int64_t)H * P;
  const float* dt_bh = p.dt + (int64_t)b * L * H + h;
  const float* al_bh = p.alpha + b * p.as0 + h * p.as2;
  const float* lm_bh = p.lambda ? p.lambda + b * p.ls0 + h * p.ls2 : nullptr;
  const float* rl_bh = p.read_logit ? p.read_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const float* wl_bh = p.write_logit ? p.write_logit + ((int64_t)b * L * H + h) * M : nullptr;
  const int64_t lg_st = (int64_t)H * M;
  constexpr int E16 = 16 / (int)sizeof(T);
  constexpr int CPR = CW / E16;
  constexpr int XV = 64 * CPR / NT;

  // Per chunk c (in reverse order), three barriers:
  //   1. x(c), dy(c) into LDS, the weights of c (from its log-decays), the adjoint into
  //      LDS, the loads of x, dy and the logits of c - 1
  //   2. the tiles Gamma^T and H, the per-token products, the loads of the state
  //      entering c - 1, the log-decays of c - 1 (the other buffer), the loads of the
  //      controls of c - 2
  //   3. the per-(token, mode) partials, dx and the adjoint update
  //   4. the dx rows of c to global memory (bfloat16; no barrier: the next chunk
  //      writes no array this phase reads)
  // Global accesses go through buffer resources whose range ends at the chunk's last
  // valid token, with per-lane offsets fixed for the whole sequence (an offset past
  // every range where a lane has nothing to access): out-of-range loads return
  // zeros, out-of-range stores are dropped, and no loaded register is merged with a
  // default value.
  constexpr unsigned kOut = 0x80000000u;
  const unsigned xs_b = (unsigned)(H * P) * (unsigned)sizeof(T);  // bytes between tokens of x, dy, dx
  auto nv_of = [&](int c) { return c >= 0 ? max(0, min(kQ, L - c * kQ)) : 0; };
  auto span = [](int nv, int64_t stride, int64_t tail) {  // bytes of rows 0 .. nv - 1
    return nv > 0 ? (int)min(((int64_t)(nv - 1) * stride + tail), (int64_t)kOut - 1) : 0;
  };
  auto rsrc = [](const void* base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
  };
  const int xtail = (P - p0) * (int)sizeof(T);
  unsigned xoff[XV];  // byte offsets of this thread's 16-byte vectors of the x / dy / dx tiles
#pragma unroll
  for (int j = 0; j < XV; ++j) {
    const int i = tid + NT * j, t = i / CPR, col = (i - t * CPR) * E16;
    xoff[j] = (p0 + col < P) ? (unsigned)t * xs_b + (unsigned)(col * (int)sizeof(T)) : kOut;
  }
  const int wm = tid % MP;  // the mode of this thread's (token, mode) pairs (NT is a multiple of MP)
  static_assert(NT % MP == 0, "every (token, mode) pair of a thread has the same mode");
  const float wr = s_rr[wm], wlnt = s_lnt[wm];
  // without logits the scores of a token are -alpha ln tau_m, whose largest lies at the
  // smallest or the largest ln tau: the value the group reduction would find
  const float lnt_lo = group_allreduce<MP>(wm < M ? wlnt : INFINITY, [](float a, float b) { return fminf(a, b); });
  const float lnt_hi = group_allreduce<MP>(wm < M ? wlnt : -INFINITY, [](float a, float b) { return fmaxf(a, b); });

  int4 xr[XV], yr[XV];
  float dt_q = 0.0f, al_q = 1.0f, lam_q = 1.0f;  // raw controls two chunks ahead, in flight
  constexpr int NPR = (kQ * MP + NT - 1) / NT;  // (token, mode) pairs per thread: pair = t MP + m = tid + NT j
  float rlr[NPR], wlr[NPR];           // the read / write logits of this thread's pairs
  unsigned loff[NPR];
#pragma unroll
  for (int j = 0; j < NPR; ++j) {
    const int pr = tid + NT * j, t = pr / MP;
    loff[j] = (pr < kQ * MP && wm < M) ? (unsigned)(t * (H * M) + wm) * 4u : kOut;
  }
  const bool own_wl = wl_bh && wl_bh != rl_bh;  // a separate write-logit array
  auto prefetch = [&](int c) {  // x, dy and the logits of chunk c (nothing past either end)
    const int t0 = c * kQ, nv = nv_of(c);
    const int xb = span(nv, xs_b, xtail);
    const auto rx = rsrc(xg + (int64_t)t0 * xstride, xb);
    const auto ry = rsrc(yg + (int64_t)t0 * xstride, xb);
#pragma unroll
    for (int j = 0; j < XV; ++j) {
      xr[j] = __builtin_bit_cast(int4, __builtin_amdgcn_raw_buffer_load_b128(rx, xoff[j], 0, 0));
      yr[j] = __builtin_bit_cast(int4, __builtin_amdgcn_raw_buffer_load_b128(ry, xoff[j], 0, 0));
    }
    const int lb = span(nv, (int64_t)H * M * 4, (int64_t)M * 4);
    const auto rr = rsrc(rl_bh ? rl_bh + (int64_t)t0 * lg_st : p.tau, rl_bh ? lb : 0);
    const auto rw = rsrc(own_wl ? wl_bh + (int64_t)t0 * lg_st : p.tau, own_wl ? lb : 0);
#pragma unroll
    for (int j = 0; j < NPR; ++j) {
      rlr[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, loff[j], 0, 0));
      wlr[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rw, loff[j], 0, 0));
    }
  };
  auto load_controls = [&](int c) {  // lane = token; zeros outside the sequence
    const int t0 = c * kQ, nv = nv_of(c);
    const auto rd = rsrc(dt_bh + (int64_t)t0 * H, span(nv, (int64_t)H * 4, 4));
    const auto ra = rsrc(al_bh + (int64_t)t0 * p.as1, span(nv, (int64_t)p.as1 * 4, 4));
    const auto rl = rsrc(lm_bh ? lm_bh + (int64_t)t0 * p.ls1 : p.tau, lm_bh ? span(nv, (int64_t)p.ls1 * 4, 4) : 0);
    dt_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rd, (unsigned)(lane * H) * 4u, 0, 0));
    al_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ra, (unsigned)(lane * p.as1) * 4u, 0, 0));
    lam_q = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rl, (unsigned)(lane * p.ls1) * 4u, 0, 0));
  };
  auto eff_step = [&](int c) {  // the effective step of this lane's token (0 past the sequence)
    const float s_eff = lm_bh ? step_factor(lam_q, al_q) : 1.0f;
    return (lane < nv_of(c)) ? dt_q * s_eff : 0.0f;
  };
  // the state entering a chunk (kept by the forward or written by the checkpoint
  // pass), four consecutive columns per thread: element e = 4 (tid + NT q) of the
  // [MP][CW] tile, staged into LDS (rounded value and remainder) for the U products
  constexpr int S4 = (MP * CW / 4 + NT - 1) / NT;
  float4 s0q[S4];
  unsigned s0off[S4];
#pragma unroll
  for (int q = 0; q < S4; ++q) {
    const int e = 4 * (tid + NT * q), m = e / CW, col = e - m * CW;
    s0off[q] = (e < MP * CW && m < M && p0 + col < P) ? (unsigned)(m * P + p0 + col) * 4u : kOut;
  }
  auto prefetch_s0 = [&](int c) {
    const auto rs = rsrc(ck_bh + (int64_t)max(c, 0) * M * P, c >= 0 ? M * P * 4 : 0);
#pragma unroll
    for (int q = 0; q < S4; ++q)
      s0q[q] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, s0off[q], 0, 0));
  };
  // the per-(token, mode) partials of row block tb = wave & 3 (modes past M store nothing)
  const int64_t part0 = (int64_t)ps * p.Bsz * H * L + (int64_t)bh * L;  // [nps][B H L][M] row of token 0
  float dtt_c, al_c;  // the effective step and order of the current chunk (lane = token)
  load_controls(nchunks - 1);
  dtt_c = eff_step(nchunks - 1);
  al_c = al_q;
  load_controls(nchunks - 2);
  prefetch(nchunks - 1);
  prefetch_s0(nchunks - 1);
  chunk_log_decays<MP, NW>(dtt_c, s_rr, P_L + ((nchunks - 1) & 1) * 2 * SW, P_L + ((nchunks - 1) & 1) * 2 * SW + SW);
  barrier();  // the log-decays of the last chunk in LDS

  for (int c = nchunks - 1; c >= 0; --c) {
    const int t0 = c * kQ, nv = min(kQ, L - t0);
    const float* P_lh = P_L + (c & 1) * 2 * SW;
    const float* P_ll = P_lh + SW;
#pragma unroll
    for (int j = 0; j < XV; ++j) {
      const int i = tid + NT * j, t = i / CPR, col = (i - t * CPR) * E16;
      *reinterpret_cast<int4*>(Xs + t * XS + col) = xr[j];
      *reinterpret_cast<int4*>(Ys + t * XS + col) = yr[j];
    }
#pragma unroll
    for (int q = 0; q < S4; ++q) {
      const int e = 4 * (tid + NT * q), m = e / CW, col = e - m * CW;
      if (e < MP * CW) {
        const floatx4 v = {s0q[q].x, s0q[q].y, s0q[q].z, s0q[q].w};
        store4(S0H + m * GQ + col, v);
        if constexpr (kBf16) {
          floatx4 lo;
#pragma unroll
          for (int i = 0; i < 4; ++i) lo[i] = v[i] - to_f32((T)v[i]);
          store4(S0L + m * GQ + col, lo);
        }
      }
    }
    const bool over = lane < MP && lane < M && !(P_lh[(lane < MP ? lane : 0) * WQ + kQ - 1] <= kNfSafe);
    const int unsafe = (int)(__ballot(over) & ((MP >= 32) ? 0xffffffffull : ((1ull << MP) - 1)));
    // ---- per (token, mode) weights: pair = t MP + m, m = wm
#pragma unroll
    for (int j = 0; j < NPR; ++j) {
      const int pr = tid + NT * j, t = pr / MP, m = wm;
      if (pr >= kQ * MP) break;  // wave-uniform
      const float dtt = __shfl(dtt_c, t, 64), al = __shfl(al_c, t, 64);
      const bool valid = t < nv;
      const float prior = -al * wlnt;
      const float zc = (m < M) ? prior + rlr[j] : -INFINITY;
      const float zw = (m < M) ? prior + wlr[j] : -INFINITY;
      float cw;
      if (!rl_bh) {  // the scores are the priors: their maximum is known
        const float e = __expf(zc - fmaxf(-al * lnt_lo, -al * lnt_hi));
        const float sum = group_allreduce<MP>(e, [](float a, float b) { return a + b; });
        cw = valid ? e * fast_rcp(sum) : 0.0f;
      } else {
        cw = valid ? group_softmax<MP>(zc) : 0.0f;
      }
      const float ww = (rl_bh == wl_bh) ? cw : (valid ? group_softmax<MP>(zw) : 0.0f);
      const float lh = P_lh[m * WQ + t];
      const bool safe = P_lh[m * WQ + kQ - 1] <= kNfSafe;
      const float kap = one_minus_exp_neg(dtt * wr) * ww;
      float* o = W + m * WQ + t;
      o[0 * SW] = cw * fexp(-lh);
      o[1 * SW] = safe ? kap * fexp(lh) : kap;
      o[2 * SW] = kap * ell_decay(P_lh + m * WQ, P_ll + m * WQ, kQ - 1, t);
      o[3 * SW] = cw;
    }
    // the adjoint at the end of the chunk, [m][p], for its products with x
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb * 16 + lg * 4 + r;
        if (m < MP) {
          const T g = (T)G[mb][r];
          GtH[m * GQ + wave * 16 + li] = g;
          if constexpr (kBf16) GtL[m * GQ + wave * 16 + li] = (T)(G[mb][r] - to_f32(g));
        }
      }
    prefetch(c - 1);  // this chunk's x, dy and logits are consumed (before the start: nothing is read)
    prefetch_s0(c - 1);  // and its entering state
    barrier();  // x, dy, weights and the adjoint in LDS
    // ---- causal tiles: Gamma^T and the masked H = dY X^T into LDS
    for (int tile = wave; tile < 10; tile += NW) {
      const int tb = tile_row(tile), kb = tile_col(tile);
      floatx4 D = {0.f, 0.f, 0.f, 0.f};  // H over this workgroup's columns
#pragma unroll
      for (int kp = 0; kp < KP; ++kp)
        mma(D, frag_load8(Ys + (tb * 16 + li) * XS + kp * 32 + lg * 8), frag_load8(Xs + (kb * 16 + li) * XS + kp * 32 + lg * 8));
      floatx4 Gm = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < (MP + 3) / 4; ++q) {
        // mode of this lane's K slot: lg (MP / 4) + q puts the 64 lanes' [m][t] reads in distinct
        // LDS banks for 16 modes (the K order of the sum is free); < MP, a multiple of 4
        const int m = lg * (MP / 4) + q;
        const bool ok = !((unsafe >> m) & 1);
        const float vO = P_O[m * WQ + tb * 16 + li];
        const float vVt = P_Vt[m * WQ + kb * 16 + li];
        Gm = __builtin_amdgcn_mfma_f32_16x16x4f32(ok ? vO : 0.0f, ok ? vVt : 0.0f, Gm, 0, 0, 0);
      }
      if (unsafe) {
        for (int m = 0; m < MP; ++m) {
          if (!((unsafe >> m) & 1)) continue;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
            if (t >= k) Gm[r] += P_c[m * WQ + t] * P_Vt[m * WQ + k] * ell_decay(P_lh + m * WQ, P_ll + m * WQ, t, k);
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = tb * 16 + lg * 4 + r, k = kb * 16 + li;
        GT[k * GS + t] = (T)keep_if_ge(Gm[r], t, k);
        HT[t * HS + k] = keep_if_ge(D[r], t, k);
      }
    }

    // ---- per token (row block tb = wave): S0 . dy and G . x, modes as output columns; with
    // bfloat16 operands the float32 state and adjoint enter as a rounded value plus its
    // rounded remainder (two products), so that these weight gradients keep float32
    // accuracy: the step-size and order gradients are differences of their sums
    floatx4 Uk[MB], Zk[MB];
    {
      const int tb = wave & 3;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int m = mb * 16 + li;  // output column of this lane
        floatx4& U = Uk[mb];
        floatx4& Z = Zk[mb];
        U = Z = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kp = 0; kp < KP; ++kp) {
          if (doU) {
            const Frag<T> yf = frag_load8(Ys + (tb * 16 + li) * XS + kp * 32 + lg * 8);
            const Frag<T> S0f = (m < MP) ? frag_load8(S0H + m * GQ + kp * 32 + lg * 8) : frag_zero<T>();
            mma(U, yf, S0f);
            if constexpr (kBf16) {  // the remainder
              const Frag<T> S0l = (m < MP) ? frag_load8(S0L + m * GQ + kp * 32 + lg * 8) : frag_zero<T>();
              mma(U, yf, S0l);
            }
          }
          if (doZ) {
            const Frag<T> xf = frag_load8(Xs + (tb * 16 + li) * XS + kp * 32 + lg * 8);
            const Frag<T> Gf = (m < MP) ? frag_load8(GtH + m * GQ + kp * 32 + lg * 8) : frag_zero<T>();
            mma(Z, xf, Gf);
            if constexpr (kBf16) {  // the remainder
              const Frag<T> Gl = (m < MP) ? frag_load8(GtL + m * GQ + kp * 32 + lg * 8) : frag_zero<T>();
              mma(Z, xf, Gl);
            }
          }
        }
      }
    }
    // sum(dy . x) of the chunk for dD (columns past d_h and tokens past the sequence are zero)
    if (p.dD) {
      for (int i = tid; i < 64 * CW; i += NT) {
        const int t = i / CW, pcol = i - t * CW;
        dd_acc += to_f32(Xs[t * XS + pcol]) * to_f32(Ys[t * XS + pcol]);
      }
    }
    // ---- the previous chunk's per-token controls and log-decays (the other buffer)
    if (c > 0) {
      dtt_c = eff_step(c - 1);
      al_c = al_q;
      float* N_lh = P_L + ((c - 1) & 1) * 2 * SW;
      chunk_log_decays<MP, NW>(dtt_c, s_rr, N_lh, N_lh + SW);
    }
    load_controls(c - 2);
    barrier();  // Gamma^T, H and the previous log-decays in LDS
    {
      // ---- per-(token, mode) partials, tokens of row block tb = wave, modes as columns:
      //   dc_{t,m} = e^{-l_t} (S0_m . dy_t) + sum_{k<=t} H_{t,k} kappa_{k,m} e^{-(l_t - l_k)}
      //   dk_{k,m} = e^{-(l_Q - l_k)} (G_m . x_k) + sum_{t>=k} H_{t,k} c_{t,m} e^{-(l_t - l_k)}
      // with the sums as float32 matrix-core products (H kappa e^{l}, H^T c e^{-l}) for
      // the factorised modes and one exp per pair for the others
      const int tb = wave & 3;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int m = mb * 16 + li;
        const int mm = m < MP ? m : 0;
        const bool fac = m < MP && !((unsafe >> mm) & 1);
        floatx4 cI = {0.f, 0.f, 0.f, 0.f}, kI = {0.f, 0.f, 0.f, 0.f};
        // 16 tokens of K per step: four reads issued together, two accumulators
        if (doU) {
          floatx4 c1 = {0.f, 0.f, 0.f, 0.f};
          for (int k4 = 0; k4 <= tb; ++k4) {
            float a[4], bb[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int k = (k4 * 4 + u) * 4 + lg;
              a[u] = HT[(tb * 16 + li) * HS + k];
              bb[u] = fac ? P_Vt[mm * WQ + k] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < 4; u += 2) {
              cI = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u], bb[u], cI, 0, 0, 0);
              c1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u + 1], bb[u + 1], c1, 0, 0, 0);
            }
          }
          cI += c1;
        }
        if (doZ) {
          floatx4 k1 = {0.f, 0.f, 0.f, 0.f};
          for (int t4 = tb; t4 < 4; ++t4) {
            float a[4], bb[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int t = (t4 * 4 + u) * 4 + lg;
              a[u] = HT[t * HS + tb * 16 + li];
              bb[u] = fac ? P_O[mm * WQ + t] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < 4; u += 2) {
              kI = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u], bb[u], kI, 0, 0, 0);
              k1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u + 1], bb[u + 1], k1, 0, 0, 0);
            }
          }
          kI += k1;
        }
        const bool direct = m < M && ((unsafe >> mm) & 1);
        const float* lhm = P_lh + mm * WQ;
        const float* llm = P_ll + mm * WQ;
        const int pb = span(nv, (int64_t)M * 4, (int64_t)M * 4);
        const unsigned po = (m < M) ? (unsigned)((tb * 16 + lg * 4) * M + m) * 4u : kOut;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb * 16 + lg * 4 + r;
          const unsigned pi = po + (unsigned)(r * M) * 4u;  // token t, mode m of [nps][B H L][M]
          if (doU) {
            const float ea = fexp(-lhm[t]);
            float dc = ea * Uk[mb][r];
            if (!direct) dc += ea * cI[r];
            else
              for (int k = 0; k <= t; ++k) dc += HT[t * HS + k] * P_Vt[mm * WQ + k] * ell_decay(lhm, llm, t, k);
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, dc), rsrc(wk.dcp + (part0 + t0) * M, pb), pi, 0, 0);
          }
          if (doZ) {
            const float dk = ell_decay(lhm, llm, kQ - 1, t) * Zk[mb][r];
            float dki = 0.0f;
            if (!direct) dki = fexp(lhm[t]) * kI[r];
            else
              for (int t2 = t; t2 < 64; ++t2) dki += HT[t2 * HS + t] * P_c[mm * WQ + t2] * ell_decay(lhm, llm, t2, t);
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, dk), rsrc(wk.dkp + (part0 + t0) * M, pb), pi, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, dki), rsrc(wk.dkip + (part0 + t0) * M, pb), pi, 0, 0);
          }
        }
      }
    }

    if (active) {
      // ---- dx: inter (weights x adjoint, K = modes), intra Gamma^T dY (K = t' >= t), skip term
      Frag<T> Gf;  // the adjoint as a B operand: slot s < 4 mode 4 lg + s, s >= 4 mode 16 + 4 lg + s - 4
#pragma unroll
      for (int s = 0; s < 4; ++s) frag_set(Gf, s, G[0][s]);
#pragma unroll
      for (int s = 0; s < 4; ++s) frag_set(Gf, 4 + s, MB > 1 ? G[MB - 1][s] : 0.0f);
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        const int t = tb * 16 + li;
        floatx4 Y = {0.f, 0.f, 0.f, 0.f};
        Frag<T> Vf;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const int m0 = lg * 4 + s, m1 = 16 + lg * 4 + s;
          frag_set(Vf, s, (m0 < MP) ? P_vq[m0 * WQ + t] : 0.0f);
          frag_set(Vf, 4 + s, (MB > 1 && m1 < MP) ? P_vq[m1 * WQ + t] : 0.0f);
        }
        mma(Y, Vf, Gf);
#pragma unroll
        for (int kk = tb / 2; kk < 2; ++kk)
          mma(Y, frag_load8(GT + t * GS + kk * 32 + lg * 8), frag_load_rows(Ys, XS, kk * 32 + lg * 8, wave * 16));
        float yv[4];
        col4_rows(Ys, XS, tb * 16 + lg * 4, wave * 16, yv);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tr = tb * 16 + lg * 4 + r;
          const float v = Y[r] + Dh * yv[r];
          if constexpr (kBf16) {
            DX[tr * XS + wave * 16 + li] = (T)v;
          } else {
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, (float)v), rsrc(dxg + (int64_t)t0 * xstride, span(nv, xs_b, xtail)),
                                                  pc < P ? (unsigned)tr * xs_b + (unsigned)(wave * 16 + li) * 4u : kOut, 0, 0);
          }
        }
      }
      // ---- adjoint update G <- e^{-l_Q} G + (c e^{-l})^T dY, rows m, column pc
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mb * 16 + lg * 4 + r;
          G[mb][r] *= (m < MP) ? fexp(-P_lh[(m < MP ? m : 0) * WQ + kQ - 1]) : 0.0f;
        }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const Frag<T> by = frag_load_rows(Ys, XS, kt * 32 + lg * 8, wave * 16);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int m = mb * 16 + li;
          Frag<T> Of;
          if (m < MP) {
            const float* po = P_O + m * WQ + kt * 32 + lg * 8;
            const float4 v0 = *reinterpret_cast<const float4*>(po);
            const float4 v1 = *reinterpret_cast<const float4*>(po + 4);
            frag_set(Of, 0, v0.x);
            frag_set(Of, 1, v0.y);
            frag_set(Of, 2, v0.z);
            frag_set(Of, 3, v0.w);
            frag_set(Of, 4, v1.x);
            frag_set(Of, 5, v1.y);
            frag_set(Of, 6, v1.z);
            frag_set(Of, 7, v1.w);
          } else {
            Of = frag_zero<T>();
          }
          mma(G[mb], Of, by);
        }
      }
    }
    barrier();  // dx rows in LDS; every array of this chunk is consumed
    if constexpr (kBf16) {
      const auto rdx = rsrc(dxg + (int64_t)t0 * xstride, span(nv, xs_b, xtail));
#pragma unroll
      for (int j = 0; j < XV; ++j) {
        const int i = tid + NT * j, t = i / CPR, col = (i - t * CPR) * E16;
        const int4 v = *reinterpret_cast<const int4*>(DX + t * XS + col);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4_t, v), rdx, xoff[j], 0, 0);
      }
    }
  }

  // ---- the adjoint of the state before token 0, and the initial-state term
  // <S_init, dS_init> per mode over this workgroup's columns
  if (p.dinit_state && active) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb * 16 + lg * 4 + r;
        if (m < M && pc < P) p.dinit_state[sbase + (int64_t)m * P + pc] = G[mb][r];
      }
  }
  __syncthreads();  // red is free again
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = mb * 16 + lg * 4 + r;
      const float ip = (p.init_state && active && m < M && pc < P) ? p.init_state[sbase + (int64_t)m * P + pc] * G[mb][r]
                                                                    : 0.0f;
      const float v = group_allreduce<16>(ip, [](float x, float y) { return x + y; });
      if (li == 0 && m < MP) red[wave][m] = v;
    }

  // ---- per-workgroup total of sum(dy . x)
  redD[tid] = dd_acc;
  __syncthreads();
  if (tid < MP && tid < M) wk.I[((int64_t)ps * p.Bsz * H + bh) * M + tid] = red_sum(tid);
  if (tid == 0) {
    float s = 0.f;
    for (int i = 0; i < NT; ++i) s += redD[i];
    wk.dDp[(int64_t)ps * p.Bsz * H + bh] = s;
  }
}

// Columns of d_h per workgroup: 128 for head dims above 128, else 64; the backward
// with 32 modes keeps 64 (LDS).
int nfree_cols(const ScanParams& p) { return p.P > 128 ? 128 : 64; }
int nfree_bwd_cols(const ScanParams& p) { return (p.P > 128 && p.M <= 16) ? 128 : 64; }

// The forward pass (CKPT: the checkpoint pass of the backward) in workgroups of NW
// waves, 16 NW columns each.
template <typename T, int MP, bool CKPT, int NW, int NH = 1>
hipError_t launch_nfree_fwd_nw(const ScanParams& p, float* ckpt, hipStream_t stream) {
  constexpr int CW = 16 * (NW / NH);
  const unsigned blocks = (unsigned)((int64_t)p.Bsz * p.H * ((p.P + CW - 1) / CW));
  hipLaunchKernelGGL((frac_nfree_fwd_kernel<T, MP, CKPT, NW, NH>), dim3(blocks), dim3(64 * NW), 0, stream, p, ckpt);
  return hipGetLastError();
}

// Head dims above 128: the outputs in 16 waves over 128 columns (two per 16
// columns, one per half of the chunk's tokens), the checkpoint pass (no outputs)
// in 8; float32 inputs with 32 modes in 4 over 64 columns (LDS).
template <typename T, int MP, bool CKPT>
hipError_t launch_nfree_fwd(const ScanParams& p, float* ckpt, hipStream_t stream) {
  if (nfree_cols(p) == 128) {
    if constexpr (CKPT) {
      return launch_nfree_fwd_nw<T, MP, CKPT, 8>(p, ckpt, stream);
    } else if constexpr (MP <= 16) {
      const unsigned blocks = (unsigned)((int64_t)p.Bsz * p.H * ((p.P + 127) / 128));
      if (ckpt)
        hipLaunchKernelGGL((frac_nfree_fwd_split_kernel<T, MP, true>), dim3(blocks), dim3(1024), 0, stream, p, ckpt);
      else
        hipLaunchKernelGGL((frac_nfree_fwd_split_kernel<T, MP, false>), dim3(blocks), dim3(1024), 0, stream, p, ckpt);
      return hipGetLastError();
    } else if constexpr (sizeof(T) == 4) {
      return launch_nfree_fwd_nw<T, MP, CKPT, 4>(p, ckpt, stream);
    } else {
      return launch_nfree_fwd_nw<T, MP, CKPT, 16, 2>(p, ckpt, stream);
    }
  }
  return launch_nfree_fwd_nw<T, MP, CKPT, 4>(p, ckpt, stream);
}

template <typename T>
hipError_t launch_nfree_t(const ScanParams& p, hipStream_t stream) {
  if (p.M <= 4) return launch_nfree_fwd<T, 4, false>(p, p.chunk_states, stream);
  if (p.M <= 8) return launch_nfree_fwd<T, 8, false>(p, p.chunk_states, stream);
  if (p.M <= 16) return launch_nfree_fwd<T, 16, false>(p, p.chunk_states, stream);
  return launch_nfree_fwd<T, 32, false>(p, p.chunk_states, stream);
}

struct NfLayout {
  size_t ckpt, F, I, dDp, tiles, dcp, dkp, dkip, total;
};

NfLayout nfree_layout(const ScanParams& p) {
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  const int cw = nfree_bwd_cols(p);
  const size_t bh = (size_t)p.Bsz * p.H, nps = (p.P + cw - 1) / cw, nch = (p.L + kQ - 1) / kQ;
  NfLayout l{};
  l.ckpt = 0;
  l.F = up(sizeof(float) * bh * (nch + 1) * p.M * p.P);
  l.I = l.F + up(sizeof(float) * nps * bh * p.M);
  l.dDp = l.I + up(sizeof(float) * nps * bh * p.M);
  l.tiles = l.dDp + up(sizeof(float) * nps * bh);
  l.dcp = l.tiles + up(grad_tiles_bytes(p));
  l.dkp = l.dcp + up(sizeof(float) * nps * bh * p.L * p.M);
  l.dkip = l.dkp + up(sizeof(float) * nps * bh * p.L * p.M);
  l.total = l.dkip + up(sizeof(float) * nps * bh * p.L * p.M);
  return l;
}

template <typename T, int MP>
hipError_t launch_nfree_bwd_mp(const ScanParams& p, void* ws, hipStream_t stream) {
  const NfLayout l = nfree_layout(p);
  unsigned char* base = reinterpret_cast<unsigned char*>(ws);
  NfWork wk;
  // the chunk states: the caller's, from its forward, or this backward's own first pass
  float* ck = p.chunk_states ? p.chunk_states : reinterpret_cast<float*>(base + l.ckpt);
  wk.ckpt = ck;
  wk.F = reinterpret_cast<float*>(base + l.F);
  wk.I = reinterpret_cast<float*>(base + l.I);
  wk.dDp = reinterpret_cast<float*>(base + l.dDp);
  wk.dcp = reinterpret_cast<float*>(base + l.dcp);
  wk.dkp = reinterpret_cast<float*>(base + l.dkp);
  wk.dkip = reinterpret_cast<float*>(base + l.dkip);
  hipError_t e = hipSuccess;
  if (!p.chunk_states && (e = launch_nfree_fwd<T, MP, true>(p, ck, stream)) != hipSuccess) return e;
  const int cw = nfree_bwd_cols(p), nps = (p.P + cw - 1) / cw;
  const unsigned blocks = (unsigned)((int64_t)p.Bsz * p.H * nps);
  constexpr bool kWide = MP <= 16;  // an 8-wave instance fits the LDS
  if constexpr (kWide) {
    if (cw == 128) hipLaunchKernelGGL((frac_nfree_bwd_kernel<T, MP, 8>), dim3(blocks), dim3(512), 0, stream, p, wk);
    else hipLaunchKernelGGL((frac_nfree_bwd_kernel<T, MP, 4>), dim3(blocks), dim3(256), 0, stream, p, wk);
  } else {
    hipLaunchKernelGGL((frac_nfree_bwd_kernel<T, MP, 4>), dim3(blocks), dim3(256), 0, stream, p, wk);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  GradInputs gi;
  gi.dc = wk.dcp;
  gi.dk = wk.dkp;
  gi.dki = wk.dkip;
  gi.ndc = gi.ndk = gi.ndki = nps;
  gi.F = wk.F;
  gi.nF = nps;
  gi.I = wk.I;
  gi.nI = nps;
  gi.dDp = wk.dDp;
  gi.nD = nps;
  grad_tiles_at(p, base + l.tiles, gi);
  return launch_grad_finish(p, gi, stream);
}

template <typename T>
hipError_t launch_nfree_bwd_t(const ScanParams& p, void* ws, hipStream_t stream) {
  if (p.M <= 4) return launch_nfree_bwd_mp<T, 4>(p, ws, stream);
  if (p.M <= 8) return launch_nfree_bwd_mp<T, 8>(p, ws, stream);
  if (p.M <= 16) return launch_nfree_bwd_mp<T, 16>(p, ws, stream);
  return launch_nfree_bwd_mp<T, 32>(p, ws, stream);
}

}  // namespace

size_t nfree_bwd_workspace(const ScanParams& p) {
  if (p.Bsz == 0 || p.L == 0) return 0;
  return nfree_layout(p).total;
}

hipError_t launch_nfree_bwd(const ScanParams& p, void* ws, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  return p.io_bf16 ? launch_nfree_bwd_t<bf16>(p, ws, stream) : launch_nfree_bwd_t<float>(p, ws, stream);
}

hipError_t launch_nfree_fwd(const ScanParams& p, hipStream_t stream) {
  if (p.Bsz == 0 || p.L == 0) return hipSuccess;
  return p.io_bf16 ? launch_nfree_t<bf16>(p, stream) : launch_nfree_t<float>(p, stream);
}

}  // namespace frac
