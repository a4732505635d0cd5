// Phase 3 of Alg. 1 on gfx950: CRT reconstruction of the exact integer,
// removal of the power-of-two scaling with ONE rounding (the paper's "one
// rounded conversion" of the multi-limb integer), and the native-FP64
// fallback for flagged rows of A / columns of B (Alg. 1, "fall back to
// native FP64 on the offending rows"; the numerical contract's item (vi)).
//
// Reconstruction.  The integer C~ in [-M/2, M/2) is unique given its r
// residues (Eq. (M-bound)), so any exact CRT algorithm yields the same bits
// as Garner's Eq. (garner).  On this VALU the direct CRT sum is cheaper than
// Garner's r(r-1)/2 dependent modular steps:
//     X = sum_i x_i W_i - q M,  W_i = (M/m_i) ((M/m_i)^-1 mod m_i),
// evaluated exactly in fp64 on 32-bit words (|x_i| <= 545, words < 2^32:
// every partial word sum is an integer below 2^46), with q = rint(sum_i x_i
// W_i/M) (error < 2^-35; an exact range check fixes the rare ambiguous case).
// The limbs are normalised to five 32-bit words (two's complement), and
// rounded once to binary64 with the exponent shift -(s_i + t_j), including
// gradual underflow and overflow.
#include "oz2_internal.h"

namespace {

constexpr int NL = OZ2_NLIMB;

// Residues of a thread's 16 outputs, as the residue buffer holds them: per
// modulus one uint4 pair = 16 int16 (output e in half e%2 of word e/2).
struct Res16 {
  uint4 lo, hi;
};

template <int E>
__device__ __forceinline__ int unpack(const Res16& v) {
  constexpr int wi = E >> 1;
  const uint32_t wd = wi == 0 ? v.lo.x : wi == 1 ? v.lo.y : wi == 2 ? v.lo.z : wi == 3 ? v.lo.w
                    : wi == 4 ? v.hi.x : wi == 5 ? v.hi.y : wi == 6 ? v.hi.z : v.hi.w;
  return (E & 1) ? (int)(int16_t)(wd >> 16) : (int)(int16_t)(wd & 0xFFFFu);
}

// Exact integer of output E of the 16 from its r centred residues: 5 words,
// two's complement, little endian.
template <int R, int E>
__device__ __forceinline__ void crt_words(const Oz2Const& c, const Res16 (&x)[OZ2_MAXR],
                                          uint32_t (&w)[NL]) {
  double S[NL];
#pragma unroll
  for (int j = 0; j < NL; ++j) S[j] = 0.0;
  double f = 0.0;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const double xi = (double)unpack<E>(x[i]);
#pragma unroll
    for (int j = 0; j < NL; ++j) S[j] = fma(xi, c.W[i][j], S[j]);
    f = fma(xi, c.wfrac[i], f);
  }
  const double q = rint(f);
#pragma unroll
  for (int j = 0; j < NL; ++j) S[j] = fma(-q, c.Ml[j], S[j]);
  // normalise: limbs 0..NL-2 into [0, 2^32), carries upward (all exact)
#pragma unroll
  for (int j = 0; j < NL - 1; ++j) {
    double cy = floor(S[j] * 0x1p-32);
    S[j] = fma(-cy, 0x1p32, S[j]);
    S[j + 1] += cy;
  }
  // the fp64 estimate of X/M is ambiguous only within 2^-35 of +-1/2
  double d = f - q;
  if (fabs(d) > 0.49999) {
    // exact range check, X in [-floor(M/2), ceil(M/2) - 1]:
    //   P = X - M + floor(M/2) >= 0  <=>  X >= ceil(M/2)   -> X -= M
    //   N = X + floor(M/2) < 0       <=>  X < -floor(M/2)  -> X += M
    // (the sign of a normalised limb vector is the sign of its top limb)
    double P[NL], N[NL];
#pragma unroll
    for (int j = 0; j < NL; ++j) { P[j] = S[j] - c.Ml[j] + c.Mhalf[j]; N[j] = S[j] + c.Mhalf[j]; }
#pragma unroll
    for (int j = 0; j < NL - 1; ++j) {
      double cp = floor(P[j] * 0x1p-32); P[j] = fma(-cp, 0x1p32, P[j]); P[j + 1] += cp;
      double cn = floor(N[j] * 0x1p-32); N[j] = fma(-cn, 0x1p32, N[j]); N[j + 1] += cn;
    }
    if (P[NL - 1] >= 0.0) {
#pragma unroll
      for (int j = 0; j < NL; ++j) S[j] -= c.Ml[j];
    } else if (N[NL - 1] < 0.0) {
#pragma unroll
      for (int j = 0; j < NL; ++j) S[j] += c.Ml[j];
    }
#pragma unroll
    for (int j = 0; j < NL - 1; ++j) {
      double cy = floor(S[j] * 0x1p-32);
      S[j] = fma(-cy, 0x1p32, S[j]);
      S[j + 1] += cy;
    }
  }
#pragma unroll
  for (int j = 0; j < NL - 1; ++j) w[j] = (uint32_t)S[j];
  w[NL - 1] = (uint32_t)(int32_t)S[NL - 1];
}

__device__ __forceinline__ uint32_t word_at(const uint32_t (&w)[NL], int i) {
  uint32_t r = 0;
#pragma unroll
  for (int j = 0; j < NL; ++j) r = (i == j) ? w[j] : r;
  return r;
}

// RN-even binary64 value of X * 2^-e for the 160-bit two's-complement X.
__device__ __forceinline__ double round_scaled(uint32_t (&w)[NL], int e) {
  const bool neg = (int32_t)w[NL - 1] < 0;
  if (neg) {                      // magnitude: two's complement negate
    uint32_t carry = 1;
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      uint32_t v = ~w[j] + carry;
      carry = (carry && v == 0) ? 1u : 0u;
      w[j] = v;
    }
  }
  int h = -1;
#pragma unroll
  for (int j = 0; j < NL; ++j) h = w[j] ? j : h;
  if (h < 0) return 0.0;         // exact zero is +0.0
  const int tb = 32 * h + (32 - __clz((int)word_at(w, h)));   // X in [2^(tb-1), 2^tb)
  const int E = tb - 1 - e;                                   // unbiased exponent of the result
  int p = 53;
  if (E < -1022) p = 53 - (-1022 - E);                        // subnormal precision
  double r;
  if (p < 0) {
    r = 0.0;                       // below half the smallest subnormal
  } else {
    const int sh = tb - p;         // bits below position sh are rounded off
    unsigned long long mant;
    if (sh <= 0) {
      mant = ((unsigned long long)w[1] << 32) | w[0];   // X < 2^53: exact
      r = ldexp((double)mant, -e);
    } else {
      const int wi = sh >> 5, bo = sh & 31;
      unsigned long long lo = ((unsigned long long)word_at(w, wi + 1) << 32) | word_at(w, wi);
      unsigned long long top = word_at(w, wi + 2);
      mant = (lo >> bo) | (bo ? (top << (64 - bo)) : 0ull);
      // round bit = bit sh-1; sticky = bits below sh-1
      const int rb = sh - 1;
      const int rwi = rb >> 5, rbo = rb & 31;
      const uint32_t rw = word_at(w, rwi);
      const bool round = (rw >> rbo) & 1u;
      bool sticky = (rw & ((1u << rbo) - 1u)) != 0u;
#pragma unroll
      for (int j = 0; j < NL; ++j) sticky |= (j < rwi) && (w[j] != 0u);
      if (round && (sticky || (mant & 1ull))) mant += 1ull;
      r = ldexp((double)mant, sh - e);
    }
  }
  return neg ? -r : r;
}

// Thread per (tile, wave, 32x32 block, lane): 16 outputs of column col,
// rows row + 8(e/4) + (e%4), e = 0..15 -- the residue GEMM's accumulator order
// (wave w owns rows (w>>2)*128 + 32x, columns (w&3)*64 + 32y of the tile).
__device__ __forceinline__ void out_coords(int mp, size_t gid, int& row, int& col, size_t& roff) {
  const int ntm = mp / OZ2_TILE;
  const size_t tile = gid >> 12;                  // 4096 threads per 256x256 tile
  const int q = (int)(gid & 4095);
  const int lane = q & 63, blk = q >> 6;          // blk = (w*4 + x)*2 + y
  const int y = blk & 1, x = (blk >> 1) & 3, w = blk >> 3;
  const int tm = (int)(tile % ntm), tn = (int)(tile / ntm);
  row = tm * OZ2_TILE + (w >> 2) * 128 + x * 32 + 4 * (lane >> 5);
  col = tn * OZ2_TILE + (w & 3) * 64 + y * 32 + (lane & 31);
  roff = tile * (OZ2_TILE * OZ2_TILE) + (size_t)q * 16;
}

template <int R>
__device__ __forceinline__ void load_residues(const int16_t* __restrict__ res, size_t plane,
                                              size_t roff, Res16 (&x)[OZ2_MAXR]) {
#pragma unroll
  for (int i = 0; i < OZ2_MAXR; ++i) {
    if (i < R) {
      const uint4* p = reinterpret_cast<const uint4*>(res + (size_t)i * plane + roff);
      x[i].lo = p[0];
      x[i].hi = p[1];
    } else {
      x[i].lo = x[i].hi = make_uint4(0u, 0u, 0u, 0u);
    }
  }
}

// one output of the 16 held by a thread: reconstruct, rescale, store
template <int R, int E>
__device__ __forceinline__ void finish_one(const Oz2Const& c, const Oz2Dims& d,
                                           const Res16 (&x)[OZ2_MAXR], int row, int tj,
                                           const int32_t* __restrict__ sA,
                                           const uint32_t* __restrict__ fA, bool acc, bool nofb,
                                           double* out) {
  const int i = row + 8 * (E >> 2) + (E & 3);
  if (i >= d.m) return;
  if (!nofb && (fA[i] & (OZ2_T1 | OZ2_T2))) return;
  uint32_t w[NL];
  crt_words<R, E>(c, x, w);
  const double v = round_scaled(w, sA[i] + tj);
  out[i] = acc ? out[i] + v : v;
}

template <int R, int E>
struct Finish {
  __device__ __forceinline__ static void run(const Oz2Const& c, const Oz2Dims& d,
                                             const Res16 (&x)[OZ2_MAXR], int row, int tj,
                                             const int32_t* __restrict__ sA,
                                             const uint32_t* __restrict__ fA, bool acc, bool nofb,
                                             double* out) {
    finish_one<R, E>(c, d, x, row, tj, sA, fA, acc, nofb, out);
    Finish<R, E + 1>::run(c, d, x, row, tj, sA, fA, acc, nofb, out);
  }
};
template <int R>
struct Finish<R, 16> {
  __device__ __forceinline__ static void run(const Oz2Const&, const Oz2Dims&,
                                             const Res16 (&)[OZ2_MAXR], int, int,
                                             const int32_t* __restrict__,
                                             const uint32_t* __restrict__, bool, bool, double*) {}
};

template <int R>
__global__ void __launch_bounds__(256)
k_reconstruct(Oz2Const c, Oz2Dims d, const int16_t* __restrict__ res,
              const int32_t* __restrict__ sA, const int32_t* __restrict__ tB,
              const uint32_t* __restrict__ fA, const uint32_t* __restrict__ fB, double* C, int ldc) {
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  int row, col;
  size_t roff;
  out_coords(d.mp, gid, row, col, roff);
  if (col >= d.n || row >= d.m) return;
  const bool acc = (d.flags & 1u) != 0;        // OZ2_ACCUMULATE
  const bool nofb = (d.flags & 8u) != 0;       // OZ2_NO_FALLBACK
  const bool force = (d.flags & 16u) != 0;     // OZ2_FORCE_FALLBACK
  const uint32_t fc = fB[col];
  if (!nofb && (force || (fc & (OZ2_T1 | OZ2_T2)))) return;
  const int tj = tB[col];
  Res16 x[OZ2_MAXR];
  load_residues<R>(res, (size_t)d.mp * d.np, roff, x);
  double* out = C + (size_t)col * ldc;
  Finish<R, 0>::run(c, d, x, row, tj, sA, fA, acc, nofb, out);
}

template <int R, int E>
struct IntOut {
  __device__ __forceinline__ static void run(const Oz2Const& c, const Oz2Dims& d,
                                             const Res16 (&x)[OZ2_MAXR], int row, int col,
                                             uint32_t* out) {
    const int i = row + 8 * (E >> 2) + (E & 3);
    if (i < d.m) {
      uint32_t w[NL];
      crt_words<R, E>(c, x, w);
      uint32_t* o = out + ((size_t)col * d.m + i) * NL;
#pragma unroll
      for (int q = 0; q < NL; ++q) o[q] = w[q];
    }
    IntOut<R, E + 1>::run(c, d, x, row, col, out);
  }
};
template <int R>
struct IntOut<R, 16> {
  __device__ __forceinline__ static void run(const Oz2Const&, const Oz2Dims&,
                                             const Res16 (&)[OZ2_MAXR], int, int, uint32_t*) {}
};

template <int R>
__global__ void __launch_bounds__(256)
k_integers(Oz2Const c, Oz2Dims d, const int16_t* __restrict__ res, uint32_t* out) {
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  int row, col;
  size_t roff;
  out_coords(d.mp, gid, row, col, roff);
  if (col >= d.n || row >= d.m) return;
  Res16 x[OZ2_MAXR];
  load_residues<R>(res, (size_t)d.mp * d.np, roff, x);
  IntOut<R, 0>::run(c, d, x, row, col, out);
}

// Compaction of flagged rows / columns into index lists (order irrelevant:
// every flagged entry is computed independently and deterministically).
__global__ void k_fallback_lists(Oz2Dims d, const uint32_t* __restrict__ fA,
                                 const uint32_t* __restrict__ fB, int* counters, int* listA,
                                 int* listB) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  const bool force = (d.flags & 16u) != 0;
  if (idx < d.m) {
    if (force || (fA[idx] & (OZ2_T1 | OZ2_T2))) listA[atomicAdd(counters + 0, 1)] = idx;
  } else if (idx < d.m + d.n) {
    const int j = idx - d.m;
    if (!force && (fB[j] & (OZ2_T1 | OZ2_T2))) listB[atomicAdd(counters + 1, 1)] = j;
  }
}

// Native FP64 for flagged entries: one FMA per k in ascending k.  A
// grid-stride loop over the device-side counts, so the launch needs no host
// synchronisation and every wave exits when the list is exhausted.
__global__ void __launch_bounds__(256)
k_fallback(Oz2Dims d, const double* __restrict__ A, int lda, const double* __restrict__ B, int ldb,
           double* C, int ldc, const int* __restrict__ counters, const int* __restrict__ listA,
           const int* __restrict__ listB, const uint32_t* __restrict__ fA) {
  const size_t na = (size_t)counters[0], nb = (size_t)counters[1];
  const size_t itemsA = na * (size_t)d.n, total = itemsA + nb * (size_t)d.m;
  const bool acc = (d.flags & 1u) != 0;
  const bool force = (d.flags & 16u) != 0;
  for (size_t it = (size_t)blockIdx.x * blockDim.x + threadIdx.x; it < total;
       it += (size_t)gridDim.x * blockDim.x) {
    int i, j;
    if (it < itemsA) {
      i = listA[it / d.n];
      j = (int)(it % d.n);
    } else {
      const size_t u = it - itemsA;
      j = listB[u / d.m];
      i = (int)(u % d.m);
      if (force || (fA[i] & (OZ2_T1 | OZ2_T2))) continue;   // done as a flagged row
    }
    const double* a = A + i;
    const double* b = B + (size_t)j * ldb;
    double s = 0.0;
    for (int l = 0; l < d.k; ++l) s = fma(a[(size_t)l * lda], b[l], s);
    double* o = C + i + (size_t)j * ldc;
    *o = acc ? *o + s : s;
  }
}

__global__ void k_fill(double* C, int m, int n, int ldc) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)m * n) return;
  const size_t j = idx / m, i = idx % m;
  C[i + j * ldc] = 0.0;
}

template <int R>
void launch_reconstruct_r(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                          double* C, int ldc, hipStream_t s) {
  const size_t threads = (size_t)d.mp * d.np / 16;
  hipLaunchKernelGGL(k_reconstruct<R>, dim3((unsigned)(threads / 256)), dim3(256), 0, s, c, d,
                     (const int16_t*)(ws + L.res), (const int32_t*)(ws + L.sA),
                     (const int32_t*)(ws + L.tB), (const uint32_t*)(ws + L.flagsA),
                     (const uint32_t*)(ws + L.flagsB), C, ldc);
}

template <int R>
void launch_integers_r(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                       uint32_t* out, hipStream_t s) {
  const size_t threads = (size_t)d.mp * d.np / 16;
  hipLaunchKernelGGL(k_integers<R>, dim3((unsigned)(threads / 256)), dim3(256), 0, s, c, d,
                     (const int16_t*)(ws + L.res), out);
}

#define OZ2_R_SWITCH(FN, ...)                 \
  switch (c.r) {                              \
    case 8: FN<8>(__VA_ARGS__); break;        \
    case 9: FN<9>(__VA_ARGS__); break;        \
    case 10: FN<10>(__VA_ARGS__); break;      \
    case 11: FN<11>(__VA_ARGS__); break;      \
    case 12: FN<12>(__VA_ARGS__); break;      \
    case 13: FN<13>(__VA_ARGS__); break;      \
    case 14: FN<14>(__VA_ARGS__); break;      \
    case 15: FN<15>(__VA_ARGS__); break;      \
    case 16: FN<16>(__VA_ARGS__); break;      \
    default: return hipErrorInvalidValue;     \
  }

}  // namespace

hipError_t oz2_launch_reconstruct(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                                  uint8_t* ws, double* C, int ldc, hipStream_t s) {
  OZ2_R_SWITCH(launch_reconstruct_r, d, L, c, ws, C, ldc, s)
  return hipGetLastError();
}

hipError_t oz2_launch_integers(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                               uint8_t* ws, uint32_t* out, hipStream_t s) {
  OZ2_R_SWITCH(launch_integers_r, d, L, c, ws, out, s)
  return hipGetLastError();
}


hipError_t oz2_launch_fallback(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, const double* A,
                               int lda, const double* B, int ldb, double* C, int ldc,
                               hipStream_t s) {
  const unsigned lb = (unsigned)((d.m + d.n + 255) / 256);
  hipLaunchKernelGGL(k_fallback_lists, dim3(lb), dim3(256), 0, s, d,
                     (const uint32_t*)(ws + L.flagsA), (const uint32_t*)(ws + L.flagsB),
                     (int*)(ws + L.counters), (int*)(ws + L.listA), (int*)(ws + L.listB));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_fallback, dim3(1024), dim3(256), 0, s, d, A, lda, B, ldb, C, ldc,
                     (const int*)(ws + L.counters), (const int*)(ws + L.listA),
                     (const int*)(ws + L.listB), (const uint32_t*)(ws + L.flagsA));
  return hipGetLastError();
}

hipError_t oz2_launch_fill(double* C, int m, int n, int ldc, hipStream_t s) {
  const size_t total = (size_t)m * n;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, C, m, n, ldc);
  return hipGetLastError();
}
