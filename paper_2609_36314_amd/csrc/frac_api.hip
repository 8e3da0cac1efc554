// frac_api.hip -- the C ABI declared in include/frac.h: argument validation,
// error reporting and dispatch to the kernel launchers.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>

#include "frac.h"
#include "frac_kernels.h"

// Device scratch of frac_scan_fwd_noalloc: one copy per GPU, held from the library's
// first use on that GPU until the process ends.  In host code `scratch` names a
// host-side stand-in; the device address comes from hipGetSymbolAddress.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

thread_local std::string g_last_error;

frac_status fail(frac_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

frac_status ok() {
  g_last_error.clear();
  return FRAC_OK;
}

bool aligned16(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int next_tile_n(int64_t n) {
  int t = 16;
  while (t < n) t <<= 1;
  return t;
}

// Validates the sizes common to every entry point and fills the size fields of p.
frac_status fill_shape(const frac_shape* sh, frac::ScanParams& p) {
  if (!sh) return fail(FRAC_ERR_INVALID_ARG, "shape is NULL");
  if (sh->batch < 0 || sh->seqlen < 0) return fail(FRAC_ERR_INVALID_ARG, "batch and seqlen must be >= 0");
  if (sh->nheads < 1 || sh->headdim < 1 || sh->dstate < 1 || sh->ngroups < 1 || sh->nmodes < 1)
    return fail(FRAC_ERR_INVALID_ARG, "nheads, headdim, dstate, ngroups and nmodes must be >= 1");
  if (sh->nheads % sh->ngroups != 0)
    return fail(FRAC_ERR_INVALID_ARG, "nheads (%lld) is not a multiple of ngroups (%lld)", (long long)sh->nheads,
                (long long)sh->ngroups);
  if (sh->io_dtype != FRAC_F32 && sh->io_dtype != FRAC_BF16)
    return fail(FRAC_ERR_INVALID_ARG, "io_dtype %d is not a frac_dtype", (int)sh->io_dtype);
  if (sh->chunk != 0 && sh->chunk != 64) return fail(FRAC_ERR_UNSUPPORTED, "chunk %lld: only 64 (or 0 = auto) is built", (long long)sh->chunk);
  if (sh->nmodes > 32) return fail(FRAC_ERR_UNSUPPORTED, "nmodes %lld > 32", (long long)sh->nmodes);
  if ((sh->dstate != 1 && sh->dstate % 8) || sh->dstate > 128)
    return fail(FRAC_ERR_UNSUPPORTED, "dstate %lld: must be 1 or a multiple of 8 and <= 128", (long long)sh->dstate);
  const int pmax = sh->dstate == 1 ? 256 : 128;  // the form without B/C takes wider heads
  if (sh->headdim % 8 || sh->headdim > pmax)
    return fail(FRAC_ERR_UNSUPPORTED, "headdim %lld: must be a multiple of 8 and <= %d", (long long)sh->headdim,
                pmax);
  const int64_t lim = (int64_t)1 << 30;
  if (sh->batch > lim || sh->seqlen > lim || sh->nheads > lim || sh->batch * sh->nheads > lim)
    return fail(FRAC_ERR_UNSUPPORTED, "sizes beyond 2^30");
  p.Bsz = (int)sh->batch;
  p.L = (int)sh->seqlen;
  p.H = (int)sh->nheads;
  p.P = (int)sh->headdim;
  p.N = (int)sh->dstate;
  p.G = (int)sh->ngroups;
  p.M = (int)sh->nmodes;
  p.Mall = p.M;
  p.PP = (p.P + 15) / 16 * 16;
  p.Pst = p.P;
  p.NP = next_tile_n(p.N);
  p.io_bf16 = sh->io_dtype == FRAC_BF16;
  return FRAC_OK;
}

// The chunked scan keeps one 64-column tile of x per chunk in LDS (headdim <= 64)
// and its share of the state in registers (nmodes <= 8).
// The tiles of 64 tokens are addressed with 32-bit byte offsets: 64 rows of x
// (H P elements apart) and of B, C (G N elements apart) must span < 2 GiB.
frac_status check_scan_shape(const frac::ScanParams& p, const char* what, bool) {
  if (p.N == 1) {  // the form without B/C (B = C = 1): headdim <= 256, up to 32 modes
    if (p.P > 256) return fail(FRAC_ERR_UNSUPPORTED, "%s: headdim %d > 256 is not built", what, p.P);
    const int64_t es = p.io_bf16 ? 2 : 4;
    if (64 * (int64_t)p.H * p.P * es >= ((int64_t)1 << 31))
      return fail(FRAC_ERR_UNSUPPORTED, "%s: nheads * headdim too large", what);
    return FRAC_OK;
  }
  if (p.P > 128) return fail(FRAC_ERR_UNSUPPORTED, "%s: headdim %d > 128 is not built", what, p.P);
  const int64_t es = p.io_bf16 ? 2 : 4, lim = (int64_t)1 << 31;
  if (64 * (int64_t)p.H * p.P * es >= lim || 64 * (int64_t)p.G * p.N * es >= lim)
    return fail(FRAC_ERR_UNSUPPORTED, "%s: nheads * headdim or ngroups * dstate too large", what);
  return FRAC_OK;
}

frac_status fill_fwd(const frac_fwd_args* a, frac::ScanParams& p, bool need_outputs) {
  if (!a) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  if (!a->x || !a->dt || !a->alpha || !a->tau)
    return fail(FRAC_ERR_INVALID_ARG, "x, dt, alpha and tau are required");
  if (p.N == 1 ? (a->Bm || a->Cm) : (!a->Bm || !a->Cm))
    return fail(FRAC_ERR_INVALID_ARG, "Bm and Cm are required for dstate > 1 and must be NULL for dstate 1");
  if (need_outputs && !a->y) return fail(FRAC_ERR_INVALID_ARG, "y is required");
  if (a->chunk_states && p.N != 1)
    return fail(FRAC_ERR_UNSUPPORTED, "chunk_states are kept for the form without B/C (dstate 1) only");
  if (!aligned16(a->x) || !aligned16(a->Bm) || !aligned16(a->Cm) || !aligned16(a->init_state) ||
      !aligned16(a->chunk_states) || (need_outputs && (!aligned16(a->y) || !aligned16(a->final_state))))
    return fail(FRAC_ERR_INVALID_ARG, "x, Bm, Cm, y and the state arrays must be 16-byte aligned");
  p.x = a->x;
  p.dt = a->dt;
  p.Bm = a->Bm;
  p.Cm = a->Cm;
  p.alpha = a->alpha;
  p.as0 = a->alpha_stride[0];
  p.as1 = a->alpha_stride[1];
  p.as2 = a->alpha_stride[2];
  p.lambda = a->lambda;
  p.ls0 = a->lambda ? a->lambda_stride[0] : 0;
  p.ls1 = a->lambda ? a->lambda_stride[1] : 0;
  p.ls2 = a->lambda ? a->lambda_stride[2] : 0;
  p.read_logit = a->read_logit;
  p.write_logit = a->write_logit;
  p.tau = a->tau;
  p.D = a->D;
  p.init_state = a->init_state;
  p.y = need_outputs ? a->y : nullptr;
  p.final_state = need_outputs ? a->final_state : nullptr;
  p.chunk_states = a->chunk_states;
  return FRAC_OK;
}

// final_state for an empty sequence: the initial state (or zeros).
__global__ void copy_or_zero_kernel(float* dst, const float* src, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src ? src[i] : 0.0f;
}

frac_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(FRAC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

// ------------------------------------------------------- parameter construction

namespace {

frac_status params_dims(const frac_shape* sh, frac::ParamsDims& d) {
  if (!sh) return fail(FRAC_ERR_INVALID_ARG, "shape is NULL");
  if (sh->batch < 0 || sh->seqlen < 0) return fail(FRAC_ERR_INVALID_ARG, "batch and seqlen must be >= 0");
  if (sh->nheads < 1 || sh->nmodes < 1) return fail(FRAC_ERR_INVALID_ARG, "nheads and nmodes must be >= 1");
  if (sh->nheads > (1 << 24) || sh->nmodes > 4096)
    return fail(FRAC_ERR_UNSUPPORTED, "nheads or nmodes too large for the parameter kernels");
  d.rows = sh->batch * sh->seqlen;
  d.H = (int)sh->nheads;
  d.M = (int)sh->nmodes;
  return ok();
}

frac_status params_inputs(const frac_params_args* a, bool need_outputs) {
  if (!a) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  if (!a->z_dt || !a->z_alpha) return fail(FRAC_ERR_INVALID_ARG, "z_dt and z_alpha are required");
  if (!(a->dt_min <= a->dt_max)) return fail(FRAC_ERR_INVALID_ARG, "dt_min must be <= dt_max");
  if (a->z_lambda && !(a->lambda_min <= a->lambda_max))
    return fail(FRAC_ERR_INVALID_ARG, "lambda_min must be <= lambda_max");
  if ((a->v_read && !a->p_read) || (a->v_write && !a->p_write))
    return fail(FRAC_ERR_INVALID_ARG, "v_read needs p_read and v_write needs p_write");
  if (need_outputs) {
    if (!a->dt || !a->alpha) return fail(FRAC_ERR_INVALID_ARG, "dt and alpha are required");
    if (!a->z_lambda != !a->lambda) return fail(FRAC_ERR_INVALID_ARG, "z_lambda and lambda go together");
    if (!a->v_read != !a->read_logit || !a->v_write != !a->write_logit)
      return fail(FRAC_ERR_INVALID_ARG, "v_read / read_logit and v_write / write_logit go together");
  }
  return ok();
}

}  // namespace

// ------------------------------------------------------------- convolution

namespace {

frac_status conv_dims(const frac_shape* sh, int64_t channels, int width, frac::ConvDims& d) {
  if (!sh) return fail(FRAC_ERR_INVALID_ARG, "shape is NULL");
  if (sh->batch < 0 || sh->seqlen < 0) return fail(FRAC_ERR_INVALID_ARG, "batch and seqlen must be >= 0");
  if (sh->seqlen > (1ll << 30)) return fail(FRAC_ERR_UNSUPPORTED, "seqlen too large");
  if (sh->io_dtype != FRAC_F32 && sh->io_dtype != FRAC_BF16)
    return fail(FRAC_ERR_INVALID_ARG, "io_dtype %d is not a frac_dtype", (int)sh->io_dtype);
  if (channels < 8 || channels % 8 || channels > (1ll << 24))
    return fail(FRAC_ERR_UNSUPPORTED, "channels %lld: must be a positive multiple of 8", (long long)channels);
  if (width < 1 || width > 4) return fail(FRAC_ERR_UNSUPPORTED, "width %d: 1..4 is built", width);
  d.rows = sh->batch * sh->seqlen;
  d.L = (int)sh->seqlen;
  d.C = (int)channels;
  d.K = width;
  d.bf16_io = sh->io_dtype == FRAC_BF16;
  return ok();
}

frac_status gnorm_dims(const frac_shape* sh, int64_t channels, int64_t group, frac::GnormDims& d) {
  if (!sh) return fail(FRAC_ERR_INVALID_ARG, "shape is NULL");
  if (sh->batch < 0 || sh->seqlen < 0) return fail(FRAC_ERR_INVALID_ARG, "batch and seqlen must be >= 0");
  if (sh->io_dtype != FRAC_F32 && sh->io_dtype != FRAC_BF16)
    return fail(FRAC_ERR_INVALID_ARG, "io_dtype %d is not a frac_dtype", (int)sh->io_dtype);
  if (channels < 8 || channels % 8 || channels > 4096)
    return fail(FRAC_ERR_UNSUPPORTED, "channels %lld: a multiple of 8 up to 4096 is built", (long long)channels);
  const int64_t nvg = group / 8;
  if (group < 8 || group % 8 || channels % group || (nvg & (nvg - 1)))
    return fail(FRAC_ERR_UNSUPPORTED, "group %lld: a multiple of 8 dividing channels, group / 8 a power of two",
                (long long)group);
  d.rows = sh->batch * sh->seqlen;
  d.C = (int)channels;
  d.group = (int)group;
  d.bf16_io = sh->io_dtype == FRAC_BF16;
  return ok();
}

}  // namespace

extern "C" {

const char* frac_status_string(frac_status s) {
  switch (s) {
    case FRAC_OK: return "FRAC_OK";
    case FRAC_ERR_INVALID_ARG: return "FRAC_ERR_INVALID_ARG: invalid argument";
    case FRAC_ERR_UNSUPPORTED: return "FRAC_ERR_UNSUPPORTED: size or option not supported";
    case FRAC_ERR_WORKSPACE: return "FRAC_ERR_WORKSPACE: workspace missing or too small";
    case FRAC_ERR_HIP: return "FRAC_ERR_HIP: HIP runtime error";
  }
  return "unknown frac_status";
}

const char* frac_last_error(void) { return g_last_error.c_str(); }

frac_status frac_default_tau(int M, double tau_min, double tau_max, float* out) {
  if (M < 1 || !(tau_min > 0.0) || !(tau_max >= tau_min) || !out)
    return fail(FRAC_ERR_INVALID_ARG, "frac_default_tau: need M >= 1, 0 < tau_min <= tau_max, out != NULL");
  if (M == 1) {
    out[0] = (float)tau_min;
    return ok();
  }
  const double lr = log(tau_max / tau_min);
  for (int m = 0; m < M; ++m) out[m] = (float)(tau_min * exp(lr * (double)m / (double)(M - 1)));
  out[M - 1] = (float)tau_max;
  return ok();
}

frac_status frac_chunk_states_size(const frac_shape* shape, size_t* bytes) {
  if (!bytes) return fail(FRAC_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = 0;
  frac::ScanParams p{};
  frac_status s = fill_shape(shape, p);
  if (s == FRAC_OK) s = check_scan_shape(p, "frac_chunk_states_size", false);
  if (s != FRAC_OK) return s;
  if (p.N != 1) return fail(FRAC_ERR_UNSUPPORTED, "chunk_states are kept for the form without B/C (dstate 1) only");
  const int64_t nchunks = ((int64_t)p.L + 63) / 64;
  *bytes = sizeof(float) * (size_t)p.Bsz * p.H * (size_t)(nchunks + 1) * p.M * p.P;
  return ok();
}

size_t frac_scan_workspace_size(const frac_shape* shape, int backward) {
  frac::ScanParams p{};
  if (fill_shape(shape, p) != FRAC_OK || check_scan_shape(p, "frac_scan_workspace_size", backward) != FRAC_OK) return 0;
  if (p.N == 1) return backward ? frac::nfree_bwd_workspace(p) : 0;  // the form without B/C
  return backward ? frac::scan_bwd_workspace(p) : frac::scan_fwd_workspace(p);
}

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device

// The current device's copy of the static scratch, looked up once per device.
frac_status static_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "frac_scan_fwd_noalloc: hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(FRAC_ERR_UNSUPPORTED, "frac_scan_fwd_noalloc: device %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return hip_status(e != hipSuccess ? e : hipErrorInvalidSymbol,
                                                   "frac_scan_fwd_noalloc: hipGetSymbolAddress(scratch)");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return FRAC_OK;
}

// frac_scan_fwd with either the caller's workspace or (use_static) the static scratch.
frac_status scan_fwd_impl(const frac_shape* shape, const frac_fwd_args* args, void* ws, size_t ws_bytes,
                          void* stream, bool use_static) {
  const char* name = use_static ? "frac_scan_fwd_noalloc" : "frac_scan_fwd";
  frac::ScanParams p{};
  frac_status s = fill_shape(shape, p);
  if (s == FRAC_OK) s = check_scan_shape(p, name, false);
  if (s != FRAC_OK) return s;
  if (p.Bsz == 0) return ok();
  if (!args) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (p.L == 0) {
    if (args->chunk_states && p.N != 1)
      return fail(FRAC_ERR_UNSUPPORTED, "chunk_states are kept for the form without B/C (dstate 1) only");
    const int64_t n = (int64_t)p.Bsz * p.H * p.M * p.N * p.P;
    // [B H][1][M][P]: the single slot of an empty sequence is its final state
    for (float* dst : {args->final_state, args->chunk_states}) {
      if (!dst) continue;
      hipLaunchKernelGGL(copy_or_zero_kernel, dim3(256), dim3(256), 0, st, dst, args->init_state, n);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return hip_status(e, "frac_scan_fwd (empty sequence)");
    }
    return ok();
  }
  s = fill_fwd(args, p, true);
  if (s != FRAC_OK) return s;
  if (p.N == 1) return hip_status(frac::launch_nfree_fwd(p, st), "frac_scan_fwd launch");
  const size_t need = frac::scan_fwd_workspace(p);
  if (use_static) {
    if (need > kStaticScratchBytes)
      return fail(FRAC_ERR_WORKSPACE, "frac_scan_fwd_noalloc: this shape needs %zu bytes of scratch, the static "
                  "scratch holds %zu (use frac_scan_fwd with a workspace)", need, kStaticScratchBytes);
    ws = nullptr;
    ws_bytes = need;
    if (need && (s = static_scratch(&ws)) != FRAC_OK) return s;
  } else if (need && (!ws || ws_bytes < need)) {
    return fail(FRAC_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  }
  return hip_status(frac::launch_scan_fwd(p, ws, ws_bytes, st), use_static ? "frac_scan_fwd_noalloc launch"
                                                                           : "frac_scan_fwd launch");
}

}  // namespace

frac_status frac_scan_fwd(const frac_shape* shape, const frac_fwd_args* args, void* ws, size_t ws_bytes,
                          void* stream) {
  return scan_fwd_impl(shape, args, ws, ws_bytes, stream, false);
}

frac_status frac_scan_fwd_noalloc(const frac_shape* shape, const frac_fwd_args* args, void* stream) {
  return scan_fwd_impl(shape, args, nullptr, 0, stream, true);
}

size_t frac_scan_fwd_noalloc_limit(void) { return kStaticScratchBytes; }

frac_status frac_scan_bwd(const frac_shape* shape, const frac_bwd_args* args, void* ws, size_t ws_bytes,
                          void* stream) {
  frac::ScanParams p{};
  frac_status s = fill_shape(shape, p);
  if (s == FRAC_OK) s = check_scan_shape(p, "frac_scan_bwd", true);
  if (s != FRAC_OK) return s;
  if (p.Bsz == 0 || p.L == 0) {
    if (args && args->dinit_state && p.Bsz > 0) {  // no tokens: the initial state is the final state
      const int64_t n = (int64_t)p.Bsz * p.H * p.M * p.N * p.P;
      hipLaunchKernelGGL(copy_or_zero_kernel, dim3(256), dim3(256), 0,
                         reinterpret_cast<hipStream_t>(stream), args->dinit_state, args->d_final_state, n);
      const frac_status e = hip_status(hipGetLastError(), "frac_scan_bwd (empty)");
      if (e != FRAC_OK) return e;
    }
    if (args && args->dD && p.Bsz >= 0) {
      hipLaunchKernelGGL(copy_or_zero_kernel, dim3(1), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                         args->dD, (const float*)nullptr, (int64_t)p.H);
      return hip_status(hipGetLastError(), "frac_scan_bwd (empty)");
    }
    return ok();
  }
  if (!args) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  s = fill_fwd(&args->fwd, p, false);
  if (s != FRAC_OK) return s;
  if (!args->dy || !args->dx || !args->ddt)
    return fail(FRAC_ERR_INVALID_ARG, "dy, dx and ddt are required");
  if (p.N == 1 ? (args->dBm || args->dCm) : (!args->dBm || !args->dCm))
    return fail(FRAC_ERR_INVALID_ARG, "dBm and dCm are required for dstate > 1 and must be NULL for dstate 1");
  if (!aligned16(args->dy) || !aligned16(args->dx) || !aligned16(args->dBm) || !aligned16(args->dCm) ||
      !aligned16(args->d_final_state))
    return fail(FRAC_ERR_INVALID_ARG, "dy, dx, dBm, dCm and d_final_state must be 16-byte aligned");
  p.dy = args->dy;
  p.d_final_state = args->d_final_state;
  p.dx = args->dx;
  p.ddt = args->ddt;
  p.dBm = args->dBm;
  p.dCm = args->dCm;
  p.dD = args->fwd.D ? args->dD : nullptr;
  p.dalpha = args->dalpha;
  p.dlambda = args->dlambda;
  p.dread_logit = args->dread_logit;
  p.dwrite_logit = args->dwrite_logit;
  p.dinit_state = args->dinit_state;
  const size_t need = p.N == 1 ? frac::nfree_bwd_workspace(p) : frac::scan_bwd_workspace(p);
  if (need && (!ws || ws_bytes < need))
    return fail(FRAC_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  if (p.N == 1) return hip_status(frac::launch_nfree_bwd(p, ws, reinterpret_cast<hipStream_t>(stream)),
                                  "frac_scan_bwd launch");
  return hip_status(frac::launch_scan_bwd(p, ws, ws_bytes, reinterpret_cast<hipStream_t>(stream)),
                    "frac_scan_bwd launch");
}

frac_status frac_decode_step(const frac_shape* shape, const frac_step_args* a, void* stream) {
  frac::ScanParams p{};
  frac_status s = fill_shape(shape, p);
  if (s != FRAC_OK) return s;
  if (shape->seqlen != 1) return fail(FRAC_ERR_INVALID_ARG, "frac_decode_step: shape.seqlen must be 1");
  if (p.Bsz == 0) return ok();
  if (!a) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  if (!a->x || !a->dt || !a->alpha || !a->tau || !a->state || !a->y)
    return fail(FRAC_ERR_INVALID_ARG, "x, dt, alpha, tau, state and y are required");
  if (p.N == 1 ? (a->Bm || a->Cm) : (!a->Bm || !a->Cm))
    return fail(FRAC_ERR_INVALID_ARG, "Bm and Cm are required for dstate > 1 and must be NULL for dstate 1");
  if (!aligned16(a->state)) return fail(FRAC_ERR_INVALID_ARG, "state must be 16-byte aligned");
  p.x = a->x;
  p.dt = a->dt;
  p.Bm = a->Bm;
  p.Cm = a->Cm;
  p.alpha = a->alpha;
  p.as0 = a->alpha_stride[0];
  p.as1 = a->alpha_stride[1];
  p.lambda = a->lambda;
  p.ls0 = a->lambda ? a->lambda_stride[0] : 0;
  p.ls1 = a->lambda ? a->lambda_stride[1] : 0;
  p.read_logit = a->read_logit;
  p.write_logit = a->write_logit;
  p.tau = a->tau;
  p.D = a->D;
  p.y = a->y;
  return hip_status(frac::launch_decode_step(p, a->state, reinterpret_cast<hipStream_t>(stream)),
                    "frac_decode_step launch");
}


frac_status frac_params_fwd(const frac_shape* shape, const frac_params_args* a, void* stream) {
  frac::ParamsDims d{};
  frac_status s = params_dims(shape, d);
  if (s != FRAC_OK) return s;
  if (d.rows == 0) return ok();
  if ((s = params_inputs(a, true)) != FRAC_OK) return s;
  return hip_status(frac::launch_params_fwd(d, *a, reinterpret_cast<hipStream_t>(stream)), "frac_params_fwd launch");
}

size_t frac_params_workspace_size(const frac_shape* shape) {
  frac::ParamsDims d{};
  if (params_dims(shape, d) != FRAC_OK) return 0;
  return frac::params_workspace(d.H);
}

frac_status frac_params_bwd(const frac_shape* shape, const frac_params_bwd_args* a, void* ws, size_t ws_bytes,
                            void* stream) {
  frac::ParamsDims d{};
  frac_status s = params_dims(shape, d);
  if (s != FRAC_OK) return s;
  if (!a) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  if (d.rows == 0) {  // nothing to read: the sums are zero
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (a->ddt_bias) hipLaunchKernelGGL(copy_or_zero_kernel, dim3(1), dim3(256), 0, st, a->ddt_bias, nullptr, (int64_t)d.H);
    if (a->dp_read) hipLaunchKernelGGL(copy_or_zero_kernel, dim3(1), dim3(64), 0, st, a->dp_read, nullptr, (int64_t)1);
    if (a->dp_write) hipLaunchKernelGGL(copy_or_zero_kernel, dim3(1), dim3(64), 0, st, a->dp_write, nullptr, (int64_t)1);
    return hip_status(hipGetLastError(), "frac_params_bwd (empty)");
  }
  if ((s = params_inputs(&a->fwd, false)) != FRAC_OK) return s;
  const size_t need = frac_params_workspace_size(shape);
  if (!ws || ws_bytes < need)
    return fail(FRAC_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  return hip_status(frac::launch_params_bwd(d, *a, reinterpret_cast<float*>(ws), reinterpret_cast<hipStream_t>(stream)),
                    "frac_params_bwd launch");
}

frac_status frac_conv_fwd(const frac_shape* shape, const frac_conv_args* a, void* stream) {
  if (!a) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  frac::ConvDims d{};
  frac_status s = conv_dims(shape, a->channels, a->width, d);
  if (s != FRAC_OK) return s;
  if (d.rows == 0) return ok();
  if (!a->x || !a->w || !a->y) return fail(FRAC_ERR_INVALID_ARG, "x, w and y are required");
  if (!aligned16(a->x) || !aligned16(a->y)) return fail(FRAC_ERR_INVALID_ARG, "x and y must be 16-byte aligned");
  return hip_status(frac::launch_conv_fwd(d, *a, reinterpret_cast<hipStream_t>(stream)), "frac_conv_fwd launch");
}

size_t frac_conv_workspace_size(const frac_shape* shape, int64_t channels, int width) {
  frac::ConvDims d{};
  if (conv_dims(shape, channels, width, d) != FRAC_OK) return 0;
  return frac::conv_workspace(d.C, d.K);
}

frac_status frac_conv_bwd(const frac_shape* shape, const frac_conv_bwd_args* a, void* ws, size_t ws_bytes,
                          void* stream) {
  if (!a) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  frac::ConvDims d{};
  frac_status s = conv_dims(shape, a->fwd.channels, a->fwd.width, d);
  if (s != FRAC_OK) return s;
  if (d.rows == 0) {  // no tokens: the sums are zero
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (a->dw) hipLaunchKernelGGL(copy_or_zero_kernel, dim3(16), dim3(256), 0, st, a->dw, nullptr, (int64_t)d.C * d.K);
    if (a->dbias) hipLaunchKernelGGL(copy_or_zero_kernel, dim3(16), dim3(256), 0, st, a->dbias, nullptr, (int64_t)d.C);
    return hip_status(hipGetLastError(), "frac_conv_bwd (empty)");
  }
  if (!a->fwd.x || !a->fwd.w || !a->dy || !a->dx) return fail(FRAC_ERR_INVALID_ARG, "x, w, dy and dx are required");
  if (!aligned16(a->fwd.x) || !aligned16(a->dy) || !aligned16(a->dx))
    return fail(FRAC_ERR_INVALID_ARG, "x, dy and dx must be 16-byte aligned");
  const size_t need = frac::conv_workspace(d.C, d.K);
  if ((a->dw || a->dbias) && (!ws || ws_bytes < need))
    return fail(FRAC_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  return hip_status(frac::launch_conv_bwd(d, *a, reinterpret_cast<float*>(ws), reinterpret_cast<hipStream_t>(stream)),
                    "frac_conv_bwd launch");
}

frac_status frac_gnorm_fwd(const frac_shape* shape, const frac_gnorm_args* a, void* stream) {
  if (!a) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  frac::GnormDims d{};
  frac_status s = gnorm_dims(shape, a->channels, a->group, d);
  if (s != FRAC_OK) return s;
  if (!(a->eps >= 0.0f)) return fail(FRAC_ERR_INVALID_ARG, "eps must be >= 0");
  if (d.rows == 0) return ok();
  if (!a->x || !a->z || !a->weight || !a->y) return fail(FRAC_ERR_INVALID_ARG, "x, z, weight and y are required");
  if (!aligned16(a->x) || !aligned16(a->z) || !aligned16(a->y))
    return fail(FRAC_ERR_INVALID_ARG, "x, z and y must be 16-byte aligned");
  return hip_status(frac::launch_gnorm_fwd(d, *a, reinterpret_cast<hipStream_t>(stream)), "frac_gnorm_fwd launch");
}

size_t frac_gnorm_workspace_size(const frac_shape* shape, int64_t channels) {
  if (!shape || channels < 8 || channels % 8 || channels > 4096) return 0;
  return frac::gnorm_workspace(channels);
}

frac_status frac_gnorm_bwd(const frac_shape* shape, const frac_gnorm_bwd_args* a, void* ws, size_t ws_bytes,
                           void* stream) {
  if (!a) return fail(FRAC_ERR_INVALID_ARG, "args is NULL");
  frac::GnormDims d{};
  frac_status s = gnorm_dims(shape, a->fwd.channels, a->fwd.group, d);
  if (s != FRAC_OK) return s;
  if (!(a->fwd.eps >= 0.0f)) return fail(FRAC_ERR_INVALID_ARG, "eps must be >= 0");
  if (d.rows == 0) {
    if (a->dweight) {
      hipLaunchKernelGGL(copy_or_zero_kernel, dim3(16), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                         a->dweight, nullptr, (int64_t)d.C);
      return hip_status(hipGetLastError(), "frac_gnorm_bwd (empty)");
    }
    return ok();
  }
  if (!a->fwd.x || !a->fwd.z || !a->fwd.weight || !a->dy || !a->dx || !a->dz)
    return fail(FRAC_ERR_INVALID_ARG, "x, z, weight, dy, dx and dz are required");
  if (!aligned16(a->fwd.x) || !aligned16(a->fwd.z) || !aligned16(a->dy) || !aligned16(a->dx) || !aligned16(a->dz))
    return fail(FRAC_ERR_INVALID_ARG, "x, z, dy, dx and dz must be 16-byte aligned");
  const size_t need = frac::gnorm_workspace(d.C);
  if (a->dweight && (!ws || ws_bytes < need))
    return fail(FRAC_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  return hip_status(frac::launch_gnorm_bwd(d, *a, reinterpret_cast<float*>(ws), reinterpret_cast<hipStream_t>(stream)),
                    "frac_gnorm_bwd launch");
}

}  // extern "C"
