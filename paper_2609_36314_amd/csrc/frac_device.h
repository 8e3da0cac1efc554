// frac_device.h -- device-side building blocks shared by the Frac scan kernels
// (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace frac {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kQ = 64;  // tokens per chunk
// Row stride (floats) of the per-(token, mode) weight arrays [mode][token] in LDS:
// 68 puts the stores of one wave (lanes = a few tokens x all modes) and the
// 16-lane row reads of 4 modes into distinct banks; rows stay 16-byte aligned.
constexpr int kWQ = kQ + 4;

// The 10 causal 16x16 tiles of a 64-token chunk in row-major lower-triangular
// order, tile = tb (tb + 1) / 2 + kb: the row block of a tile (plain arithmetic,
// so no table load sits on the path of a tile loop).
__device__ __forceinline__ int tile_row(int tile) { return (tile >= 1) + (tile >= 3) + (tile >= 6); }
__device__ __forceinline__ int tile_col(int tile) { const int tb = tile_row(tile); return tile - tb * (tb + 1) / 2; }

// A value fixed in a register at this point.  A prefetched register read after
// later memory operations have been issued makes the wave wait for those too (the
// vector-memory counter drains in order, and direct-to-LDS copies are not tracked
// by the compiler), so each chunk takes its prefetched values this way right after
// its memory wait, before it issues the next chunk's copies and loads.
__device__ __forceinline__ float pinned(float v) {
  asm volatile("" : "+v"(v));
  return v;
}

// The read / write logits of the (token, mode) pairs that a thread of an NT-thread
// workgroup forms in a chunk's weight pass (pair = t MP + m = tid + NT j), loaded
// one chunk ahead into registers: the weight pass then never waits on global
// memory (a wait there would also drain the next chunk's tile copies).  Zero for
// pairs past the chunk, absent logits, and wl when the write logits are the read
// logits (the weight pass reuses the read weights then).
// LSE (a mode block): also the two per-token log-normalizers lse[t * lse_st + {0, 1}],
// lane = token, which the weight pass takes with a lane shuffle.
template <int MP, int NT, bool LSE = false>
struct PairLogits {
  static constexpr int NPR = (kQ * MP + NT - 1) / NT;
  float rl[NPR], wl[NPR];
  float ln_c = 0.0f, ln_w = 0.0f;
  __device__ __forceinline__ void load(const float* rlp, const float* wlp, int t0, int nv, int M, int64_t stride,
                                       int tid, const float* lse = nullptr, int64_t lse_st = 0) {
#pragma unroll
    for (int j = 0; j < NPR; ++j) {
      const int pr = tid + NT * j, t = pr / MP, m = pr - t * MP;
      const bool ok = pr < kQ * MP && t < nv && m < M;
      const int64_t i = (int64_t)(t0 + t) * stride + m;
      rl[j] = (ok && rlp) ? rlp[i] : 0.0f;
      wl[j] = (ok && wlp && wlp != rlp) ? wlp[i] : 0.0f;
    }
    if constexpr (LSE) {
      const int tl = tid & 63;
      const float2 v = tl < nv ? *reinterpret_cast<const float2*>(lse + (int64_t)(t0 + tl) * lse_st) : float2{0.0f, 0.0f};
      ln_c = v.x;
      ln_w = v.y;
    }
  }
  __device__ __forceinline__ PairLogits pinned_copy() const {
    PairLogits o;
#pragma unroll
    for (int j = 0; j < NPR; ++j) {
      o.rl[j] = pinned(rl[j]);
      o.wl[j] = pinned(wl[j]);
    }
    if constexpr (LSE) {
      o.ln_c = pinned(ln_c);
      o.ln_w = pinned(ln_w);
    }
    return o;
  }
};

// ---------------------------------------------------------------- fragments
//
// A 16x16x32 matrix-core step consumes, per lane (i = lane % 16, g = lane / 16),
// eight K-slots of the A row i and eight K-slots of the B column i.  Which K index
// a slot stands for is free as long as A and B agree; every fragment below is
// built with an explicit slot -> K map and both operands of a product use the
// same map.  For float32 operands the step is issued as eight 16x16x4 products,
// slot s of lane group g going to product s.

template <typename T>
struct Frag;
template <>
struct Frag<bf16> {
  bf16x8 v;
};
template <>
struct Frag<float> {
  float v[8];
};

__device__ __forceinline__ void mma(floatx4& acc, const Frag<bf16>& a, const Frag<bf16>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}

__device__ __forceinline__ void mma(floatx4& acc, const Frag<float>& a, const Frag<float>& b) {
#pragma unroll
  for (int s = 0; s < 8; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[s], b.v[s], acc, 0, 0, 0);
}

template <typename T>
__device__ __forceinline__ Frag<T> frag_zero() {
  Frag<T> f;
#pragma unroll
  for (int s = 0; s < 8; ++s) f.v[s] = (T)0.0f;
  return f;
}

template <typename T>
__device__ __forceinline__ void frag_set(Frag<T>& f, int s, float val) {
  f.v[s] = (T)val;
}

// Eight consecutive elements at p (16-byte aligned for bf16, 32-byte for float).
__device__ __forceinline__ Frag<bf16> frag_load8(const bf16* p) {
  Frag<bf16> f;
  f.v = *reinterpret_cast<const bf16x8*>(p);
  return f;
}
__device__ __forceinline__ Frag<float> frag_load8(const float* p) {
  Frag<float> f;
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
  return f;
}

// Slots 0..3 from p0[0..3], slots 4..7 from p1[0..3]; with two = false slots
// 4..7 are zero and p1 is not read.  (No null-pointer test: comparing an LDS
// address against null miscompiles on this target.)
__device__ __forceinline__ Frag<bf16> frag_load4x2(const bf16* p0, const bf16* p1, bool two = true) {
  Frag<bf16> f;
  const bf16x4 a = *reinterpret_cast<const bf16x4*>(p0);
  bf16x4 b = bf16x4{(bf16)0.0f, (bf16)0.0f, (bf16)0.0f, (bf16)0.0f};
  if (two) b = *reinterpret_cast<const bf16x4*>(p1);
  f.v = bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return f;
}
__device__ __forceinline__ Frag<float> frag_load4x2(const float* p0, const float* p1, bool two = true) {
  Frag<float> f;
  const float4 a = *reinterpret_cast<const float4*>(p0);
  float4 b = make_float4(0.f, 0.f, 0.f, 0.f);
  if (two) b = *reinterpret_cast<const float4*>(p1);
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
  return f;
}

// ------------------------------------------------------------ io conversion

__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }
__device__ __forceinline__ float to_f32(float v) { return v; }

// Load 8 consecutive io elements from global memory as floats.
__device__ __forceinline__ void load8(const bf16* p, float* out) {
  const bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int j = 0; j < 8; ++j) out[j] = (float)v[j];
}
__device__ __forceinline__ void load8(const float* p, float* out) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
  out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
}

// Four consecutive io elements as floats (8-byte aligned for bf16, 16 for float).
__device__ __forceinline__ void load4(const bf16* p, float* out) {
  const bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
#pragma unroll
  for (int j = 0; j < 4; ++j) out[j] = (float)v[j];
}
__device__ __forceinline__ void load4(const float* p, float* out) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
}

// Store four floats as four consecutive io elements.
__device__ __forceinline__ void store4(bf16* p, const floatx4& v) {
  *reinterpret_cast<bf16x4*>(p) = bf16x4{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
}
__device__ __forceinline__ void store4(float* p, const floatx4& v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}

// Raw copy of 8 io elements global -> shared, no conversion.
__device__ __forceinline__ void copy8(bf16* dst, const bf16* src) {
  *reinterpret_cast<bf16x8*>(dst) = *reinterpret_cast<const bf16x8*>(src);
}
__device__ __forceinline__ void copy8(float* dst, const float* src) {
  reinterpret_cast<float4*>(dst)[0] = reinterpret_cast<const float4*>(src)[0];
  reinterpret_cast<float4*>(dst)[1] = reinterpret_cast<const float4*>(src)[1];
}

template <typename T>
__device__ __forceinline__ void zero8(T* dst) {
#pragma unroll
  for (int j = 0; j < 8; ++j) dst[j] = (T)0.0f;
}

// ------------------------------------------------------------- wave helpers

// Inclusive prefix sum over the 64 lanes of a wave (Hillis-Steele, fixed order).
__device__ __forceinline__ float wave_inclusive_sum(float v) {
  // within each row of 16 lanes: add the lanes 1, 2, 4, 8 places lower (zero past
  // the row start); then the last lane of row 0 (2) into row 1 (3), and lane 31
  // into rows 2 and 3
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x111, 0xF, 0xF, true));  // row_shr:1
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x112, 0xF, 0xF, true));  // row_shr:2
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x114, 0xF, 0xF, true));  // row_shr:4
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x118, 0xF, 0xF, true));  // row_shr:8
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xA, 0xF, false)); // row_bcast:15
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x143, 0xC, 0xF, false)); // row_bcast:31
  return v;
}

// The same inclusive prefix sum in float64 (each DPP move carries one half of the
// value; lanes with no source read +0.0).
template <int CTRL, int ROW_MASK, bool BOUND>
__device__ __forceinline__ double dpp_move_f64(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(b & 0xffffffffll), CTRL, ROW_MASK, 0xF, BOUND);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(b >> 32), CTRL, ROW_MASK, 0xF, BOUND);
  return __longlong_as_double(((long long)hi << 32) | (long long)(unsigned)lo);
}
__device__ __forceinline__ double wave_inclusive_sum_f64(double v) {
  v += dpp_move_f64<0x111, 0xF, true>(v);   // row_shr:1
  v += dpp_move_f64<0x112, 0xF, true>(v);   // row_shr:2
  v += dpp_move_f64<0x114, 0xF, true>(v);   // row_shr:4
  v += dpp_move_f64<0x118, 0xF, true>(v);   // row_shr:8
  v += dpp_move_f64<0x142, 0xA, false>(v);  // row_bcast:15
  v += dpp_move_f64<0x143, 0xC, false>(v);  // row_bcast:31
  return v;
}

// v plus the value of lane ^ 16 (lane ^ 32): the two halves exchanged with one
// cross-row swap, the sum formed in the same order in both lanes.
__device__ __forceinline__ float xor16_sum(float v) {
  const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}
__device__ __forceinline__ float xor32_sum(float v) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// ------------------------------------------------------- per-token controls

// Scalar-broadcast strided load: element (i0,i1,i2) at p[i0*s0 + i1*s1 + i2*s2].
__device__ __forceinline__ float strided3(const float* p, int64_t s0, int64_t s1, int64_t s2, int64_t i0,
                                          int64_t i1, int64_t i2) {
  return p[i0 * s0 + i1 * s1 + i2 * s2];
}

// softmax over the first M of MP entries (the rest get weight 0), in place.
template <int MP>
__device__ __forceinline__ void softmax_modes(float* z, int M) {
  float mx = z[0];
#pragma unroll
  for (int m = 1; m < MP; ++m)
    if (m < M) mx = fmaxf(mx, z[m]);
  float sum = 0.f;
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    z[m] = (m < M) ? expf(z[m] - mx) : 0.f;
    sum += z[m];
  }
  const float inv = 1.0f / sum;
#pragma unroll
  for (int m = 0; m < MP; ++m) z[m] *= inv;
}

// Effective step dt * lambda^(1/alpha) (eq. tau-eff).

// lambda^{1/alpha}, the factor of the effective step, held at or below 2^100 so that
// chunk sums of steps stay finite (a factor that large already decays every mode with
// tau < 2^80 to zero in float32 within one step of at least 1e-4).
__device__ __forceinline__ float step_factor(float lam, float alpha) {
  return exp2f(fminf(log2f(lam) / alpha, 100.0f));
}

__device__ __forceinline__ float effective_step(float dt, float alpha, const float* lam_ptr, float lam) {
  return lam_ptr ? dt * step_factor(lam, alpha) : dt;
}

// ------------------------------------------------- per-mode chunk log-decays
//
// The decay between tokens k <= t of one chunk in mode m is e^{-(l_{t,m} - l_{k,m})}
// with l_{t,m} the chunk-local inclusive sum of r_m dtt_j (eq. rho-beta-def-frac:
// the product of the retentions rho is the exponential of the summed exponents).
// Each exponent is capped at kCapExp first: e^{-kCapExp} is zero in float32, so a
// capped token still cuts every decay across it to exactly zero, while the sums
// stay below 64 kCapExp.  The sums are formed per mode in float64 and kept as a
// float pair (hi = float(l), lo = float(l - hi)): a difference of two such pairs
// is exact to float32 rounding for any mix of effective steps in the chunk, where
// one float32 prefix sum of dtt shared by all modes would lose the small steps
// that follow a step near 1e13.
constexpr float kCapExp = 110.0f;

// r_m dtt capped; mask is 1 where the cap is not reached (the exponent then
// depends on dtt with slope r_m, else not at all).
__device__ __forceinline__ float capped_exponent(float r, float dtt) { return fminf(r * dtt, kCapExp); }

// Wave w of an NW-wave workgroup, lane = token, forms modes w, w + NW, ... of the
// chunk (dtt_l: this lane's effective step, 0 past the chunk's valid tokens;
// s_rr: the rates, 0 for padding modes).  Writes hi / lo pairs [MP][kWQ].
template <int MP, int NW>
__device__ __forceinline__ void chunk_log_decays(float dtt_l, const float* s_rr, float* ell_hi, float* ell_lo) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int m0 = 0; m0 < MP; m0 += NW) {
    const int m = m0 + wave;
    if (m0 + NW > MP && m >= MP) break;  // wave-uniform
    const double v = wave_inclusive_sum_f64((double)capped_exponent(s_rr[m], dtt_l));
    const float hi = (float)v;
    ell_hi[m * kWQ + lane] = hi;
    ell_lo[m * kWQ + lane] = (float)(v - (double)hi);
  }
}

// l_a - l_b from two hi / lo pairs.
__device__ __forceinline__ float ell_diff(float hia, float loa, float hib, float lob) {
  return (hia - hib) + (loa - lob);
}

// e^{-(l_a - l_b)} for a >= b (entries a, b of one mode's row of the hi / lo arrays),
// the interval clamped at zero so that rounding never lifts a decay above 1.
__device__ __forceinline__ float ell_decay(const float* lh, const float* ll, int a, int b) {
  return __expf(-fmaxf(ell_diff(lh[a], ll[a], lh[b], ll[b]), 0.0f));
}

// ------------------------------------------------------- fast scalar math

// e^x through the hardware exp2 (a multiply and one transcendental).
__device__ __forceinline__ float fexp(float x) { return __expf(x); }

// 1 / x through the hardware reciprocal (one transcendental, about 1 ulp) for a
// normal, finite x: a softmax normaliser (>= 1) or a state scale (>= 2^-60).
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// 1 - e^{-x} for x >= 0 without cancellation: a short Taylor series where the
// difference is small, the subtraction elsewhere (relative error <= ~4e-6).
__device__ __forceinline__ float one_minus_exp_neg(float x) {
  const float series = x * (1.0f - x * (0.5f - x * (1.0f / 6.0f - x * (1.0f / 24.0f - x * (1.0f / 120.0f)))));
  return x < 0.0625f ? series : 1.0f - __expf(-x);
}

// softmax over the first M of MP entries with the fast exponential.
template <int MP>
__device__ __forceinline__ void softmax_fast(float* z, int M) {
  float mx = z[0];
#pragma unroll
  for (int m = 1; m < MP; ++m)
    if (m < M) mx = fmaxf(mx, z[m]);
  float sum = 0.f;
#pragma unroll
  for (int m = 0; m < MP; ++m) {
    z[m] = (m < M) ? __expf(z[m] - mx) : 0.0f;
    sum += z[m];
  }
  const float inv = fast_rcp(sum);
#pragma unroll
  for (int m = 0; m < MP; ++m) z[m] *= inv;
}

// x where row >= col, else +0: the mask is the sign of col - row - 1 spread over
// all 32 bits, so no per-lane condition registers are formed (or kept live).
__device__ __forceinline__ float keep_if_ge(float x, int row, int col) {
  return __int_as_float(__float_as_int(x) & ((col - row - 1) >> 31));
}

// One DPP row permutation of a float (every lane of the wave active).
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}

// op over each aligned group of G consecutive lanes (G a power of two <= 64),
// returned in every lane of the group, bit-identical across the group.  Groups
// up to 16 lanes use DPP: swap neighbours, swap pairs (quad permutations), then
// pair each lane with its mirror in the 8- and 16-lane rows, which at that point
// belongs to the other half and already holds that half's result; wider groups
// swap rows.
template <int G, typename Op>
__device__ __forceinline__ float group_allreduce(float v, Op op) {
  if constexpr (G >= 2) v = op(v, dpp_move<0xB1>(v));   // quad_perm [1, 0, 3, 2]
  if constexpr (G >= 4) v = op(v, dpp_move<0x4E>(v));   // quad_perm [2, 3, 0, 1]
  if constexpr (G >= 8) v = op(v, dpp_move<0x141>(v));  // row_half_mirror
  if constexpr (G >= 16) v = op(v, dpp_move<0x140>(v)); // row_mirror
  if constexpr (G >= 32) {  // the lane 16 places away, through a cross-row swap
    const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = op(__uint_as_float(s[0]), __uint_as_float(s[1]));
  }
  if constexpr (G >= 64) {
    const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = op(__uint_as_float(s[0]), __uint_as_float(s[1]));
  }
  return v;
}

// softmax across the MP consecutive lanes that hold the modes of one token (MP a
// power of two dividing 64, lane = token * MP + mode, the whole wave active);
// -inf entries get weight 0.
template <int MP>
__device__ __forceinline__ float group_softmax(float z) {
  const float mx = group_allreduce<MP>(z, [](float a, float b) { return fmaxf(a, b); });
  const float e = __expf(z - mx);
  const float sum = group_allreduce<MP>(e, [](float a, float b) { return a + b; });
  return e * fast_rcp(sum);
}

// The thread index behind an empty asm statement: values derived from it inside
// a loop body are recomputed there instead of being hoisted out of the loop and
// held (or spilled) for its whole duration.
__device__ __forceinline__ int fresh_tid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

// ------------------------------------------------ LDS fragment reads (K = rows)

typedef short v4i16 __attribute__((ext_vector_type(4)));

// Eight K-slots from a row-major LDS matrix (row stride ld elements): slot s holds
// row row0 + s of column col0 + (lane % 16).  For bfloat16 this is two transposed
// 64-bit LDS reads (ds_read_b64_tr_b16): within each 16-lane group, lane i
// addresses 4 consecutive elements of row row0 + i/4 at column col0 + 4 (i % 4),
// and lane j receives column col0 + j of the 4 rows.  row0 may differ between
// the 16-lane groups.
__device__ __forceinline__ Frag<bf16> frag_load_rows(const bf16* m, int ld, int row0, int col0, int tid = threadIdx.x) {
  const int li = tid & 15;
  const bf16* p = m + (row0 + (li >> 2)) * ld + col0 + 4 * (li & 3);
  const v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(p));
  const v4i16 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(p + 4 * ld));
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  const v8i16 ab = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  Frag<bf16> f;
  f.v = __builtin_bit_cast(bf16x8, ab);
  return f;
}
__device__ __forceinline__ Frag<float> frag_load_rows(const float* m, int ld, int row0, int col0, int tid = threadIdx.x) {
  const int li = tid & 15;
  Frag<float> f;
#pragma unroll
  for (int s = 0; s < 8; ++s) f.v[s] = m[(row0 + s) * ld + col0 + li];
  return f;
}

// Four consecutive rows row0..row0+3 of column col0 + (lane % 16), as floats
// (one transposed read for bfloat16).
__device__ __forceinline__ void col4_rows(const bf16* m, int ld, int row0, int col0, float* out, int tid = threadIdx.x) {
  const int li = tid & 15;
  const bf16* p = m + (row0 + (li >> 2)) * ld + col0 + 4 * (li & 3);
  const v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(p));
  const bf16x4 v = __builtin_bit_cast(bf16x4, a);
#pragma unroll
  for (int s = 0; s < 4; ++s) out[s] = (float)v[s];
}
__device__ __forceinline__ void col4_rows(const float* m, int ld, int row0, int col0, float* out, int tid = threadIdx.x) {
  const int li = tid & 15;
#pragma unroll
  for (int s = 0; s < 4; ++s) out[s] = m[(row0 + s) * ld + col0 + li];
}

// -------------------------------------------------- direct global -> LDS tiles

// Direct global -> LDS copy of a 64-row tile with a padded LDS row stride LDW
// (elements; LDW * sizeof(T) a multiple of 16), through a buffer resource.  A
// block of 8 waves issues KT 16-byte copies per lane; copy k of wave w fills LDS
// bytes [(8k + w) 1024, +1024), so lane l writes 16-byte chunk
// q = (8k + w) 64 + l = row * (LDW / E) + chunk of the tile.  The per-lane byte
// offsets depend on the sizes only and are computed once (init).  Chunks that are
// padding or lie past `cols`, and rows past the valid ones, get an offset past the
// resource's range: the hardware returns zeros for them.
template <typename T, int LDW>
struct DmaPlan {
  static constexpr int E = 16 / sizeof(T);
  static constexpr int CPR = LDW / E;  // 16-byte chunks per LDS row
  static constexpr int KT = (64 * CPR + 511) / 512;
  static constexpr unsigned kOut = 0x80000000u;  // >= every range handed to issue()
  unsigned off[KT];
  // gstride: elements between consecutive rows; requires 64 gstride sizeof(T) < 2^31
  __device__ __forceinline__ void init(int64_t gstride, int cols) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
    for (int k = 0; k < KT; ++k) {
      const int q = (k * 8 + wave) * 64 + lane;
      const int row = q / CPR, ch = q - row * CPR;
      off[k] = (q < 64 * CPR && ch * E < cols) ? (unsigned)((row * gstride + ch * E) * (int64_t)sizeof(T)) : kOut;
    }
  }
  // Copy the tile whose first row is at src; only the first nv rows are in range.
  // OPAQUE: pass the LDS address as a plain 32-bit offset instead of an address
  // space cast (for single-buffered tiles; some constant-folded casts of LDS
  // addresses do not compile on this target).
  template <bool OPAQUE = false>
  __device__ __forceinline__ void issue(T* lds, const T* src, int64_t gstride, int nv) const {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const long long range = (long long)nv * gstride * (long long)sizeof(T);
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)src, (short)0, (int)(range < kOut ? range : kOut), 0x00020000);
#pragma unroll
    for (int k = 0; k < KT; ++k) {
      if (k * 8 + wave >= CPR) continue;  // past the tile (uniform)
      T* dst = lds + (k * 8 + wave) * 64 * E;
      __attribute__((address_space(3))) void* l3;
      if constexpr (OPAQUE) l3 = (__attribute__((address_space(3))) void*)(uintptr_t)(uint32_t)(uintptr_t)dst;
      else l3 = (__attribute__((address_space(3))) void*)dst;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, l3, 16, (int)off[k], 0, 0, 0);
    }
  }
  // The same copy issued as an instruction the compiler does not see as an LDS
  // write: it then does not wait for the copy before every later LDS read (which it
  // must assume may alias the copy's destination), so the next chunk's copy
  // overlaps the current chunk's work.  The caller waits for it explicitly
  // (wait_vmem) before the barrier that publishes the tile.
  __device__ __forceinline__ void issue_async(T* lds, const T* src, int64_t gstride, int nv) const {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const long long range = (long long)nv * gstride * (long long)sizeof(T);
    const uint64_t a = (uint64_t)(uintptr_t)src;
    typedef int i32x4 __attribute__((ext_vector_type(4)));
    i32x4 rs;  // buffer resource: base, stride 0, byte range, raw-buffer flags
    rs[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    rs[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu));
    rs[2] = __builtin_amdgcn_readfirstlane((int)(range < kOut ? range : kOut));
    rs[3] = 0x00020000;
#pragma unroll
    for (int k = 0; k < KT; ++k) {
      if (k * 8 + wave >= CPR) continue;  // past the tile (uniform)
      const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds + (k * 8 + wave) * 64 * E));
      asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                   :
                   : "s"(m0), "v"(off[k]), "s"(rs)
                   : "memory", "m0");
    }
  }
};

// This lane's 4 io values of the C B^T tiles `wave` and `wave + 8` of one chunk
// (10 lower-triangular 16x16 tiles of 256 values, lane-major), loaded one chunk
// ahead of their use.
template <typename T>
struct TilePrefetch {
  struct alignas(4 * sizeof(T)) V {
    T e[4];
  };
  V v[2];
  __device__ __forceinline__ void load(const T* chunk_tiles, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int tile = wave + 8 * j;
      if (tile < 10) v[j] = *reinterpret_cast<const V*>(chunk_tiles + tile * 256 + lane * 4);
    }
  }
  __device__ __forceinline__ float get(int j, int r) const { return to_f32(v[j].e[r]); }
  __device__ __forceinline__ TilePrefetch pinned_copy() const {  // see pinned()
    TilePrefetch o;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      constexpr int W = sizeof(V) / 4;
      uint32_t w[W];
      __builtin_memcpy(w, &v[j], sizeof(V));
#pragma unroll
      for (int i = 0; i < W; ++i) asm volatile("" : "+v"(w[i]));
      __builtin_memcpy(&o.v[j], w, sizeof(V));
    }
    return o;
  }
};

// Wait for this wave's outstanding vector-memory operations (including the
// direct-to-LDS copies, which the compiler does not count).
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Workgroup barrier for LDS traffic: this wave's LDS accesses complete, then
// s_barrier.  Unlike __syncthreads it does not wait for outstanding global loads,
// so direct-to-LDS copies of the next tile stay in flight across it (their
// completion is awaited with wait_vmem before the barrier that publishes them).
__device__ __forceinline__ void barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace frac
