// frac_kernels.h -- host-side launch interface between the C ABI (frac_api.hip)
// and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "frac.h"

namespace frac {

// Validated problem description handed to the kernel launchers.  Sizes are the
// caller's; PP and NP are P and N rounded up to the 16-wide matrix-core tile.
struct ScanParams {
  int Bsz, L, H, P, N, G, M;
  int PP, NP;
  // Row stride of x, y, dx, dy and the P extent of the states (the caller's headdim).
  // A launch may cover P <= Pst columns of it (a column group, its pointers offset).
  int Pst;
  int col0;  // the first column of this launch's group (offsets the workspace's P-wide arrays)
  int io_bf16;
  const void* x;
  const float* dt;
  const void* Bm;
  const void* Cm;
  const float* alpha;
  int64_t as0, as1, as2;
  const float* lambda;
  int64_t ls0, ls1, ls2;
  const float* read_logit;
  const float* write_logit;
  const float* tau;
  const float* D;
  const float* init_state;
  void* y;
  float* final_state;
  // the form without B/C: [B H][nchunks + 1][M][P] the state entering each chunk, then
  // the final state; written by the forward, read by the backward in place of its own
  // checkpoint pass (NULL: not kept)
  float* chunk_states;
  // forward split into nseg sequence segments of seg_len tokens (the last shorter;
  // nseg 1: no split).  seg_state [nseg-1][B H Mall N P]: the state after each
  // segment but the last (first each segment's own end state from a zero start,
  // then the true boundary state); seg_decay [nseg-1][B H Mall]: each segment's
  // total per-mode decay e^{-sum of the capped exponents}.
  int seg_len, nseg;
  float* seg_state;
  float* seg_decay;
  // Mode blocks (more modes than one launch holds): a launch covers M modes of Mall
  // (the per-mode pointers tau, logits and states already offset to its first mode;
  // logits and states keep the strides of Mall).  lse: per token the log-normalizers
  // of the read and write softmax over all Mall modes ([B L H][2]; NULL: over the
  // launch's own modes).  y_in: float32 sum of the earlier blocks' outputs (NULL for
  // the first); y_part: float32 output of a block that is not the last (NULL: write
  // y, with the skip term).
  int Mall;
  const float* lse;
  const float* y_in;
  float* y_part;
  // backward only
  const void* dy;
  const float* d_final_state;
  void* dx;
  float* ddt;
  void* dBm;
  void* dCm;
  float* dD;
  // further gradients (each NULL = not produced)
  float* dalpha;
  float* dlambda;
  float* dread_logit;
  float* dwrite_logit;
  float* dinit_state;
};

// The launch parameters of the columns [c0, c0 + 64) of P (at most 64): the column
// count, and every pointer whose last dimension is P offset to the first column.
inline ScanParams column_group(const ScanParams& p, int c0) {
  ScanParams q = p;
  q.col0 = c0;
  q.P = p.Pst - c0 < 64 ? p.Pst - c0 : 64;
  q.PP = (q.P + 15) / 16 * 16;
  const size_t es = p.io_bf16 ? 2 : 4;
  auto off = [&](const void* v) { return v ? static_cast<const void*>(static_cast<const char*>(v) + es * c0) : v; };
  q.x = off(p.x);
  q.y = p.y ? static_cast<char*>(p.y) + es * c0 : nullptr;
  q.dy = off(p.dy);
  q.dx = p.dx ? static_cast<char*>(p.dx) + es * c0 : nullptr;
  q.init_state = p.init_state ? p.init_state + c0 : nullptr;
  q.final_state = p.final_state ? p.final_state + c0 : nullptr;
  q.d_final_state = p.d_final_state ? p.d_final_state + c0 : nullptr;
  q.dinit_state = p.dinit_state ? p.dinit_state + c0 : nullptr;
  return q;
}

// Each launcher returns hipSuccess or the launch error; `stream` may be null.
hipError_t launch_scan_fwd(const ScanParams& p, void* ws, size_t ws_bytes, hipStream_t stream);
size_t scan_fwd_workspace(const ScanParams& p);

// The per-token log-normalizers of the read and write softmax over all p.Mall modes
// (the mode blocks' weights), [B L H][2].
hipError_t launch_mode_lse(const ScanParams& p, float* lse, hipStream_t stream);

// C B^T of every chunk (causal 16x16 tiles, per-lane fragment order), shared by
// the heads of a group; `tiles` holds cb_tiles_bytes(p) bytes.
size_t cb_tiles_bytes(const ScanParams& p);
hipError_t launch_cb_tiles(const ScanParams& p, void* tiles, hipStream_t stream);

hipError_t launch_scan_bwd(const ScanParams& p, void* ws, size_t ws_bytes, hipStream_t stream);
size_t scan_bwd_workspace(const ScanParams& p);

// Control-branch parameter construction (frac_params.hip).
struct ParamsDims {
  int64_t rows;  // B * L
  int H, M;
};
hipError_t launch_params_fwd(const ParamsDims& d, const frac_params_args& a, hipStream_t stream);
constexpr int kParamsMaxBlocks = 1024;  // partial sums of the backward: 2 floats per block, H per row block
size_t params_workspace(int64_t H);
hipError_t launch_params_bwd(const ParamsDims& d, const frac_params_bwd_args& a, float* part, hipStream_t stream);

// Causal depthwise convolution of the content branch (frac_conv.hip).
struct ConvDims {
  int64_t rows;  // B * L
  int L, C, K;
  bool bf16_io;
};
constexpr int kConvMaxRowBlocks = 256;
size_t conv_workspace(int64_t C, int K);
hipError_t launch_conv_fwd(const ConvDims& d, const frac_conv_args& a, hipStream_t stream);
hipError_t launch_conv_bwd(const ConvDims& d, const frac_conv_bwd_args& a, float* ws, hipStream_t stream);

// Gated normalization of the layer output (frac_gnorm.hip).
struct GnormDims {
  int64_t rows;  // B * L
  int C, group;
  bool bf16_io;
};
constexpr int kGnormMaxRowBlocks = 1024;
size_t gnorm_workspace(int64_t C);
hipError_t launch_gnorm_fwd(const GnormDims& d, const frac_gnorm_args& a, hipStream_t stream);
hipError_t launch_gnorm_bwd(const GnormDims& d, const frac_gnorm_bwd_args& a, float* ws, hipStream_t stream);

hipError_t launch_decode_step(const ScanParams& p, float* state, hipStream_t stream);

// The layer without B/C projections (dstate 1, B = C = 1): forward scan (no
// workspace) and backward (workspace of nfree_bwd_workspace(p) bytes).
hipError_t launch_nfree_fwd(const ScanParams& p, hipStream_t stream);
size_t nfree_bwd_workspace(const ScanParams& p);
hipError_t launch_nfree_bwd(const ScanParams& p, void* ws, hipStream_t stream);

// Gradients of dt, alpha, lambda, the read / write logits and D from the
// per-(token, mode) partials of a reverse sweep (frac_grads.hip):
//   dc [ndc][B H L][M]    partials of dL/dc_{t,m}  (slot 0 may be overwritten with the sum)
//   dk [ndk][B H L][M]    partials of the inter-chunk part of dL/dkappa_{t,m} (through
//                         the adjoint carried in from the later chunks)
//   dki [ndki][B H L][M]  partials of its intra-chunk part
//   F  [nF][B H][M]     partials of <dS_final, S_final> per mode (the final-state term)
//   I  [nI][B H][M]     partials of <S_init, dS_init> per mode (the initial-state term)
//   dDp [nD][B H]       partials of sum(dy . x)
//   tileV, tileF        scratch of grad_tiles_bytes(p) bytes, placed by grad_tiles_at
// Writes p.ddt and, where non-NULL, p.dalpha, p.dlambda, p.dread_logit,
// p.dwrite_logit and p.dD.
struct GradInputs {
  float* dc;
  float* dk;
  float* dki;
  int ndc, ndk, ndki;
  int store_sums;  // set by the launcher: the first kernel writes the sums into slot 0
  const float* F;
  int nF;
  const float* I;
  int nI;
  const float* dDp;
  int nD;
  float* tileV;
  float* carry;
  int* tileF;
};
size_t grad_tiles_bytes(const ScanParams& p);
void grad_tiles_at(const ScanParams& p, void* base, GradInputs& gi);
hipError_t launch_grad_finish(const ScanParams& p, const GradInputs& gi, hipStream_t stream);

// True when a kernel variant exists for these sizes (M, N, P, dtype).
bool scan_supported(const ScanParams& p, const char** why);

}  // namespace frac
