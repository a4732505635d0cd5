// Device helpers shared by the deconstruction, reconstruction and batched
// kernels (each translation unit gets its own inline copies).
#pragma once
#include "oz2_internal.h"

namespace {

constexpr int NL = OZ2_NLIMB;

constexpr unsigned long long kAbsMask = 0x7FFFFFFFFFFFFFFFull;
constexpr unsigned long long kInfBits = 0x7FF0000000000000ull;

__device__ __forceinline__ unsigned long long abs_bits(double x) {
  return (unsigned long long)__double_as_longlong(x) & kAbsMask;
}

// frexp exponent of the finite positive double with bit pattern b (b != 0):
// x = f * 2^E with f in [1/2, 1).
__device__ __forceinline__ int exp_of_bits(unsigned long long b) {
  int e = (int)(b >> 52);
  if (e) return e - 1022;
  return (64 - __clzll((long long)b)) - 1074;
}

// 4-bit magnitude code c = ceil(16 |x| 2^-E), 0 iff x == 0, else in [1, 16].
// |x| < 2^E so c <= 16; the scaled value is exact whenever it is >= 1.
__device__ __forceinline__ float code_of(double x, int E) {
  if (x == 0.0) return 0.0f;
  double y = ceil(ldexp(fabs(x), 4 - E));
  return (float)fmax(y, 1.0);
}

__device__ __forceinline__ uint32_t pack4_fp8(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return (uint32_t)w;
}

// widths sigma = min(62, c - ceil(ell(R)/2)), ell(x) = ceil(log2 x) (0 for x <= 1)
__device__ __forceinline__ int width_of(unsigned long long R, int budget) {
  int ell = (R > 1) ? (64 - __clzll((long long)(R - 1))) : 0;
  return min(62, budget - ((ell + 1) >> 1));
}

// Centred residue of the exact integer a = ah 2^32 + al (|a| <= 2^62) modulo m:
// t = ah (2^32 mod m) + al is exact (|t| < 2^42) and congruent to a; then
// q = floor(t/m + 1/2) and d = t - q m is the centred residue in
// [-floor(m/2), ceil(m/2) - 1].  The fp64 value of t/m + 1/2 is within 2^-18
// of the true one, and the true one is never within 1/(2m) of an integer for
// odd m (t/m is never a half-integer); for m = 1024 every step is exact.  So
// the floor is always the exact one.
__device__ __forceinline__ int centred_residue(double ah, double al, double m, double c32,
                                               double dinv) {
  const double t = fma(ah, c32, al);
  const double q = floor(fma(t, dinv, 0.5));
  return (int)fma(-q, m, t);
}

// bytes p of four table entries, packed (element j in byte j)
__device__ __forceinline__ uint32_t gather_byte(uint32_t e0, uint32_t e1, uint32_t e2, uint32_t e3,
                                                uint32_t sel) {
  const uint32_t x01 = __builtin_amdgcn_perm(e1, e0, sel);
  const uint32_t x23 = __builtin_amdgcn_perm(e3, e2, sel);
  return __builtin_amdgcn_perm(x23, x01, 0x05040100u);
}

// 32-bit words of the two's complement integer in [-M/2, M/2) for r moduli
// (log2 M = 76.0, 85.0, 94.0, 102.9, 111.8, 120.8, 129.7, 138.5, 147.4 for
// r = 8..16; the host checks the same rule).
template <int R>
struct NWords {
  static constexpr int value = R <= 10 ? 3 : (R <= 13 ? 4 : 5);
};

// Residue I of the 8 a thread holds for one modulus (int16 I of the uint4).
template <int I>
__device__ __forceinline__ double res_at(const uint4& v) {
  constexpr int wi = I >> 1;
  const uint32_t wd = wi == 0 ? v.x : wi == 1 ? v.y : wi == 2 ? v.z : v.w;
  return (double)((I & 1) ? ((int32_t)wd >> 16) : (int32_t)(int16_t)(wd & 0xFFFFu));
}

// limbs j < NW-1 into [0, 2^32) with carries upward (every step exact:
// integers below 2^48)
template <int NW>
__device__ __forceinline__ void normalise(double (&S)[NW]) {
#pragma unroll
  for (int j = 0; j < NW - 1; ++j) {
    const double cy = floor(S[j] * 0x1p-32);
    S[j] = fma(-cy, 0x1p32, S[j]);
    S[j + 1] += cy;
  }
}

// The staged residue format: 8 outputs of a thread per modulus in a 96-bit
// record of three 32-bit words, output I in bits 12 I .. 12 I + 11, as
// u = x + floor(m/2) + 32 (0 <= u <= m + 64 < 2^12 for |x| <= m/2 + 32).
template <int I>
__device__ __forceinline__ uint32_t slot_bits(const uint3& v) {
  constexpr int b = 12 * I, wi = b >> 5, sh = b & 31;
  const uint32_t lo = wi == 0 ? v.x : (wi == 1 ? v.y : v.z);
  if constexpr (sh + 12 <= 32) {
    return (lo >> sh) & 0xFFFu;
  } else {
    const uint32_t hi = wi == 0 ? v.y : v.z;
    return __builtin_amdgcn_alignbit(hi, lo, sh) & 0xFFFu;
  }
}
template <int I>
__device__ __forceinline__ double slot_at(const uint3& v) {
  return (double)slot_bits<I>(v);
}

// The sums S_j = sum_i x_i W_i[j] of the direct CRT sum, from int16
// representatives (|x_i| <= 577) or from stored records (S_j starts at
// -sum_i (floor(m_i/2) + 32) W_i[j] and adds u_i W_i[j]: the same integers,
// exact at every step, every partial sum below 2^47).
template <int R, int NW, int I>
__device__ __forceinline__ void crt_sums(const Oz2Const& c, const uint4 (&x)[R], double (&S)[NW]) {
#pragma unroll
  for (int j = 0; j < NW; ++j) S[j] = 0.0;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const double xi = res_at<I>(x[i]);
#pragma unroll
    for (int j = 0; j < NW; ++j) S[j] = fma(xi, c.W[i][j], S[j]);
  }
}
template <int R, int NW, int I>
__device__ __forceinline__ void crt_sums(const Oz2Const& c, const uint3 (&x)[R], double (&S)[NW]) {
#pragma unroll
  for (int j = 0; j < NW; ++j) S[j] = -c.Kw[j];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const double ui = slot_at<I>(x[i]);
#pragma unroll
    for (int j = 0; j < NW; ++j) S[j] = fma(ui, c.W[i][j], S[j]);
  }
}

// Exact integer of output I of a thread from its R residues (int16
// representatives of magnitude <= 577, or stored records):
// NW words, two's complement, little endian.
template <int R, int NW, int I, class X>
__device__ __forceinline__ void crt_words(const Oz2Const& c, const X (&x)[R], uint32_t (&w)[NW]) {
  double S[NW];
  crt_sums<R, NW, I>(c, x, S);
  // quotient estimate q = rint(X / M) from the three top (unnormalised)
  // limbs: |S_j| < 2^46, |X/M| <= sum |x_i| < 2^14, so the estimate of X/M
  // is within 2^-36 of the true value; only within that of +-1/2 can q be
  // off by one, and an exact range check below settles those.
  double f = fma(S[NW - 2], 0x1p-32, S[NW - 1]);
  f = fma(S[NW - 3], 0x1p-64, f);
  f *= c.mtop;
  const double q = rint(f);
#pragma unroll
  for (int j = 0; j < NW; ++j) S[j] = fma(-q, c.Ml[j], S[j]);
  normalise<NW>(S);
  if (fabs(f - q) > 0.49999) {
    // exact range check, X in [-floor(M/2), ceil(M/2) - 1]:
    //   P = X - M + floor(M/2) >= 0  <=>  X >= ceil(M/2)   -> X -= M
    //   N = X + floor(M/2) < 0       <=>  X < -floor(M/2)  -> X += M
    // (the sign of a normalised limb vector is the sign of its top limb)
    double P[NW], N[NW];
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      P[j] = S[j] - c.Ml[j] + c.Mhalf[j];
      N[j] = S[j] + c.Mhalf[j];
    }
    normalise<NW>(P);
    normalise<NW>(N);
    const double adj = (P[NW - 1] >= 0.0) ? -1.0 : ((N[NW - 1] < 0.0) ? 1.0 : 0.0);
#pragma unroll
    for (int j = 0; j < NW; ++j) S[j] = fma(adj, c.Ml[j], S[j]);
    normalise<NW>(S);
  }
#pragma unroll
  for (int j = 0; j < NW - 1; ++j) w[j] = (uint32_t)S[j];
  w[NW - 1] = (uint32_t)(int32_t)S[NW - 1];
}

template <int NW>
__device__ __forceinline__ uint32_t word_at(const uint32_t (&w)[NW], int i) {
  uint32_t r = 0;
#pragma unroll
  for (int j = 0; j < NW; ++j) r = (i == j) ? w[j] : r;
  return r;
}

// RN-even value of |X| 2^-e for a nonzero magnitude whose result is
// subnormal or zero (the rare path): explicit round and sticky bits at the
// reduced precision of the subnormal range.
template <int NW>
__device__ __forceinline__ double round_subnormal(const uint32_t (&w)[NW], int tb, int e) {
  const int E = tb - 1 - e;
  const int p = 53 - (-1022 - E);   // bits kept, < 53
  if (p < 0) return 0.0;            // below half the smallest subnormal
  const int sh = tb - p;            // bits below position sh are rounded off (sh > 0)
  const int wi = sh >> 5, bo = sh & 31;
  const unsigned long long lo = ((unsigned long long)word_at(w, wi + 1) << 32) | word_at(w, wi);
  const unsigned long long top = word_at(w, wi + 2);
  unsigned long long mant = (lo >> bo) | (bo ? (top << (64 - bo)) : 0ull);
  const int rb = sh - 1;
  const int rwi = rb >> 5, rbo = rb & 31;
  const uint32_t rw = word_at(w, rwi);
  const bool round = (rw >> rbo) & 1u;
  bool sticky = (rw & ((1u << rbo) - 1u)) != 0u;
#pragma unroll
  for (int j = 0; j < NW; ++j) sticky |= (j < rwi) && (w[j] != 0u);
  if (round && (sticky || (mant & 1ull))) mant += 1ull;
  return ldexp((double)mant, sh - e);
}

// RN-even binary64 value of X 2^-e for the NW-word two's complement X.
// The top 64 bits of |X| (leading bit at bit 63) with a sticky bit OR-ed
// into bit 0 round to the same 53-bit value as |X| itself (64 > 53 + 2), and
// one fma of the two 32-bit halves performs that rounding; the power-of-two
// scaling is exact (or overflows to infinity, the correctly rounded result)
// unless the result is subnormal, which takes the explicit path.
template <int NW>
__device__ __forceinline__ double round_scaled(const uint32_t (&x)[NW], int e) {
  const uint32_t sm = (uint32_t)((int32_t)x[NW - 1] >> 31);   // all ones if X < 0
  uint32_t w[NW];
  uint32_t cy = sm & 1u;
#pragma unroll
  for (int j = 0; j < NW; ++j) {   // |X| = (X ^ sm) + (sm & 1)
    const uint32_t v = (x[j] ^ sm) + cy;
    cy = (v < cy) ? 1u : 0u;
    w[j] = v;
  }
  uint32_t P[NW];                  // prefix ORs for the sticky bit
  P[0] = w[0];
#pragma unroll
  for (int j = 1; j < NW; ++j) P[j] = P[j - 1] | w[j];
  // a, b, c: the top nonzero word and the two below it; st: OR of the rest
  uint32_t a = w[NW - 1], b = w[NW - 2], c = w[NW - 3];
  uint32_t st = NW >= 4 ? P[NW >= 4 ? NW - 4 : 0] : 0u;
  int top = NW - 1;
#pragma unroll
  for (int s = 0; s < NW - 1; ++s) {
    const bool z = (a == 0u);
    const int ni = NW - 4 - s;     // word that enters below c on a shift
    const uint32_t nxt = ni >= 0 ? w[ni >= 0 ? ni : 0] : 0u;
    const uint32_t nst = ni >= 1 ? P[ni >= 1 ? ni - 1 : 0] : 0u;
    a = z ? b : a;
    b = z ? c : b;
    c = z ? nxt : c;
    st = z ? nst : st;
    top -= z ? 1 : 0;
  }
  if (a == 0u) return 0.0;         // exact zero is +0.0
  const int lz = __clz((int)a);
  const int tb = 32 * top + 32 - lz;                  // |X| in [2^(tb-1), 2^tb)
  double v;
  if (tb - 1 - e < -1022) {
    v = round_subnormal<NW>(w, tb, e);
  } else {
    const uint32_t hi = lz ? __builtin_amdgcn_alignbit(a, b, 32 - lz) : a;
    const uint32_t lo = lz ? __builtin_amdgcn_alignbit(b, c, 32 - lz) : b;
    const uint32_t stk = ((st | (c << lz)) != 0u) ? 1u : 0u;
    v = ldexp(fma((double)hi, 0x1p32, (double)(lo | stk)), tb - 64 - e);
  }
  return sm ? -v : v;
}

// ---- the exact integer in radix-2^38 fp64 limbs --------------------------
// X = sum_l S[l] 2^(38 l) with S[l] in [0, 2^38) for l < NB - 1 after
// normalisation and S[NB - 1] signed; [-M/2, M/2) fits three limbs for
// r <= 12 (log2 M < 113) and four for r <= 16 (log2 M < 148).  Every limb
// sum is an integer below 2^53, so the fp64 arithmetic is exact: the limbs of
// W_i and M are below 2^38, |x_i| <= 577 (or u_i <= m_i + 64 from stored
// records, whose offsets' share K38 < 2^52 starts the sums), so with at most
// 16 terms every partial sum stays below 2^52, and the q M correction
// (|q| <= sum |x_i| + 1 < 2^14) keeps it below 2^53.
template <int R>
struct Limbs38 {
  static constexpr int value = R <= 12 ? 3 : 4;
};

template <int NB>
__device__ __forceinline__ void normalise38(double (&S)[NB]) {
#pragma unroll
  for (int l = 0; l < NB - 1; ++l) {
    const double cy = floor(S[l] * 0x1p-38);
    S[l] = fma(-cy, 0x1p38, S[l]);
    S[l + 1] += cy;
  }
}

// The normalised limbs as NB + 1 32-bit words of two's complement, little
// endian.  Three limbs: X = b1 2^64 + b0 with b0 = S0 + (S1 mod 2^26) 2^38
// and b1 = S2 2^12 + floor(S1 / 2^26).  Four limbs: b1 holds bits 64..127
// (the top 12 bits of S1, S2, the low 14 bits of S3) and the fifth word
// floor(S3 / 2^14).
template <int NB>
__device__ __forceinline__ void limbs38_words(const double (&S)[NB], uint32_t (&w)[NB + 1]) {
  static_assert(NB == 3 || NB == 4, "three or four limbs");
  const unsigned long long u0 = (unsigned long long)S[0], u1 = (unsigned long long)S[1];
  const unsigned long long b0 = u0 | (u1 << 38);
  w[0] = (uint32_t)b0;
  w[1] = (uint32_t)(b0 >> 32);
  if constexpr (NB == 3) {
    const long long b1 = (long long)S[2] * 4096 + (long long)(u1 >> 26);
    w[2] = (uint32_t)b1;
    w[3] = (uint32_t)((unsigned long long)b1 >> 32);
  } else {
    const unsigned long long u2 = (unsigned long long)S[2];
    const long long t = (long long)S[3];
    const unsigned long long b1 = (u1 >> 26) | (u2 << 12) | ((unsigned long long)t << 50);
    w[2] = (uint32_t)b1;
    w[3] = (uint32_t)(b1 >> 32);
    w[4] = (uint32_t)(t >> 14);
  }
}

// RN-even binary64 value of X 2^-e from normalised limbs.  With T the top
// limb: if T is in [-2^15, 2^15), H = T 2^38 + S[NB-2] is exact (|H| <= 2^53)
// and stands in for the top two limbs; with three limbs one fma then rounds
// H 2^38 + S0 once.  Otherwise |T 2^38 + S[NB-2]| >= 2^53, where binary64
// rounding boundaries fall on integers, so the limbs below can stand in as a
// sticky half: + 0.5 when any of them is nonzero rounds like X itself.  Four
// limbs apply the same test once more, to H.  The power-of-two scaling is
// exact unless the result overflows (to infinity, the correct rounding) or
// is subnormal, which takes the 32-bit word routine above.
template <int NB>
__device__ __forceinline__ double round38(const double (&S)[NB], int e) {
  static_assert(NB == 3 || NB == 4, "three or four limbs");
  double v;
  int sh;
  const double T = S[NB - 1];
  if constexpr (NB == 3) {
    if (T >= -0x1p15 && T < 0x1p15) {
      v = fma(fma(T, 0x1p38, S[1]), 0x1p38, S[0]);
      sh = 0;
    } else {
      v = fma(T, 0x1p38, S[1] + (S[0] != 0.0 ? 0.5 : 0.0));
      sh = 38;
    }
  } else {
    if (T >= -0x1p15 && T < 0x1p15) {
      const double H = fma(T, 0x1p38, S[2]);
      if (H >= -0x1p15 && H < 0x1p15) {
        v = fma(fma(H, 0x1p38, S[1]), 0x1p38, S[0]);
        sh = 0;
      } else {
        v = fma(H, 0x1p38, S[1] + (S[0] != 0.0 ? 0.5 : 0.0));
        sh = 38;
      }
    } else {
      v = fma(T, 0x1p38, S[2] + ((S[1] != 0.0 || S[0] != 0.0) ? 0.5 : 0.0));
      sh = 76;
    }
  }
  if (v == 0.0) return 0.0;        // exact zero is +0.0
  const int ev = (int)((__double_as_longlong(v) >> 52) & 0x7ff) - 1023;   // |v| >= 1
  if (ev + sh - e < -1022) {
    // subnormal result: X as 32-bit words
    uint32_t w[NB + 1];
    limbs38_words<NB>(S, w);
    return round_scaled<NB + 1>(w, e);
  }
  return ldexp(v, sh - e);
}

// X - qM with q = rint(X/M) estimated from the top two (unnormalised) limbs:
// the limbs dropped and the roundings move the estimate by less than 2^-24,
// so q may be off by one only where the estimate lies within that of +-1/2.
// Normalises, and returns whether the estimate was that close, where
// crt38_fix settles the range exactly.  mtop38 = 2^(38 (NB - 1)) / M.
template <int NB>
__device__ __forceinline__ bool crt38_reduce(const Oz2Const& c, double (&S)[NB]) {
  const double f = fma(S[NB - 2], 0x1p-38, S[NB - 1]) * c.mtop38;
  const double q = rint(f);
#pragma unroll
  for (int l = 0; l < NB; ++l) S[l] = fma(-q, c.M38[l], S[l]);
  normalise38<NB>(S);
  return fabs(f - q) > 0.49999;
}

// X in [-floor(M/2), ceil(M/2) - 1]: P = X - M + floor(M/2) >= 0 means
// X >= ceil(M/2) (subtract M); N = X + floor(M/2) < 0 means X <
// -floor(M/2) (add M); the sign of a normalised limb vector is that of its
// top limb
template <int NB>
__device__ __forceinline__ void crt38_fix(const Oz2Const& c, double (&S)[NB]) {
  double P[NB], N[NB];
#pragma unroll
  for (int l = 0; l < NB; ++l) {
    P[l] = S[l] - c.M38[l] + c.Mhalf38[l];
    N[l] = S[l] + c.Mhalf38[l];
  }
  normalise38<NB>(P);
  normalise38<NB>(N);
  const double adj = (P[NB - 1] >= 0.0) ? -1.0 : ((N[NB - 1] < 0.0) ? 1.0 : 0.0);
#pragma unroll
  for (int l = 0; l < NB; ++l) S[l] = fma(adj, c.M38[l], S[l]);
  normalise38<NB>(S);
}

// The exact integer C~ of an output as normalised radix-2^38 limbs: the
// direct CRT sum, the reduction by the quotient estimate, and the exact range
// check where the estimate is ambiguous.  (The reconstruction rounds these
// limbs; the integer query of the staged API exports them.)
template <int R, int NB>
__device__ __forceinline__ void crt38_acc(const Oz2Const& c, const double (&xi)[R],
                                          double (&S)[NB]) {
  static_assert(NB == Limbs38<R>::value, "limb count of r moduli");
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int l = 0; l < NB; ++l) S[l] = fma(xi[i], c.W38[i][l], S[l]);
}
template <int R, int NB>
__device__ __forceinline__ void crt38_sum(const Oz2Const& c, const double (&xi)[R],
                                          double (&S)[NB]) {
#pragma unroll
  for (int l = 0; l < NB; ++l) S[l] = 0.0;
  crt38_acc<R, NB>(c, xi, S);
  if (crt38_reduce<NB>(c, S)) crt38_fix<NB>(c, S);
}

// from int16 representatives (output I of the thread's eight)
template <int R, int I, int NB>
__device__ __forceinline__ void crt38_limbs(const Oz2Const& c, const uint4 (&x)[R],
                                            double (&S)[NB]) {
  double xi[R];
#pragma unroll
  for (int i = 0; i < R; ++i) xi[i] = res_at<I>(x[i]);
  crt38_sum<R, NB>(c, xi, S);
}
// from stored records: the limb sums start at -K38 (the offsets' share) and
// add u_i W38[i]: the same exact integers as from the representatives
template <int R, int I, int NB>
__device__ __forceinline__ void crt38_limbs(const Oz2Const& c, const uint3 (&x)[R],
                                            double (&S)[NB]) {
  double ui[R];
#pragma unroll
  for (int i = 0; i < R; ++i) ui[i] = slot_at<I>(x[i]);
#pragma unroll
  for (int l = 0; l < NB; ++l) S[l] = -c.K38[l];
  crt38_acc<R, NB>(c, ui, S);
  if (crt38_reduce<NB>(c, S)) crt38_fix<NB>(c, S);
}

template <int R, int I, class X>
__device__ __forceinline__ double crt38_rounded(const Oz2Const& c, const X (&x)[R], int e) {
  constexpr int NB = Limbs38<R>::value;
  double S[NB];
  crt38_limbs<R, I, NB>(c, x, S);
  return round38<NB>(S, e);
}

}  // namespace
