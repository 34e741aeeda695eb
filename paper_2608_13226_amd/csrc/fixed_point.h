// The greedy's 64-bit fixed point (Sec. 3.5, Eq. 15-16 summed exactly):
// a term v_j max(0, b_j - C) becomes floor(v_j max(0, b_j - C) 2^S) for a
// per-scene scale S, and gains and the objective are exact integer sums of
// such terms.  Shared by the greedy kernels and by the FST epilogue that
// also sums the greedy's first gains.
#pragma once

#include <hip/hip_runtime.h>

namespace cp {

// Fixed-point value of a nonnegative term: floor(t 2^S) as a 64-bit
// integer, for t 2^S < 2^62 (the scale S is chosen so that every gain and
// the objective stay below 2^62).  t 2^S is exact (a power-of-two scaling);
// its high and low 32-bit halves are taken by truncating float64 -> uint32
// conversions, the low half from the exact remainder t 2^S - high 2^32.
// Negative values and NaN give 0.  Float64 arithmetic only, no branches.
__device__ __forceinline__ long long fx(double t, int S) {
  const double y = fmax(__builtin_ldexp(t, S), 0.0);
  const unsigned h = (unsigned)(y * 0x1p-32);
  const unsigned l = (unsigned)__builtin_fma(-double(h), 0x1p32, y);
  return (long long)(((unsigned long long)h << 32) | l);
}

__device__ __forceinline__ double fx_to_double(long long g, int S) { return __builtin_ldexp(double(g), -S); }

// fx(v d, S) for many terms of one capacity v: vs = max(v 2^S, 0) is taken
// once, and for float d >= 0 the product vs d is exact (two 24-bit
// significands), so fx_scaled(vs, d) equals fx(v d, S) bit for bit with no
// scaling or clamping per term.  Returned as the unsigned 64-bit pattern, so
// that a difference of two terms is one 64-bit subtraction.
__device__ __forceinline__ double fx_scale(double v, int S) { return fmax(__builtin_ldexp(v, S), 0.0); }
__device__ __forceinline__ unsigned long long fx_scaled(double vs, float d) {
  const double y = vs * double(d);
  const unsigned h = (unsigned)(y * 0x1p-32);
  const unsigned l = (unsigned)__builtin_fma(-double(h), 0x1p32, y);
  return ((unsigned long long)h << 32) | l;
}

// fx_scaled(vs, d1) - fx_scaled(vs, d2) when both products are below 2^52
// (the incremental form's scale guarantees it for every term): floor(y) +
// 2^52 is then exact and lies in [2^52, 2^53), where the float64 bit
// pattern is that of 2^52 plus the integer floor(y), so the difference of
// the two patterns is the difference of the floors.  Four float64
// operations a term instead of seven.
__device__ __forceinline__ long long fx_diff(double vs, float d1, float d2) {
  const double a = __builtin_floor(vs * double(d1)) + 0x1p52;
  const double b = __builtin_floor(vs * double(d2)) + 0x1p52;
  return __double_as_longlong(a) - __double_as_longlong(b);
}

// fx_scaled(vs, d) as a signed integer when vs d < 2^52 (the incremental
// form's scale guarantees it): the floor plus 2^52, whose float64 bit
// pattern is that of 2^52 plus the integer, less that pattern's bias.
__device__ __forceinline__ long long fx_term(double vs, float d) {
  return __double_as_longlong(__builtin_floor(vs * double(d)) + 0x1p52) - 0x4330000000000000ll;
}

}  // namespace cp
