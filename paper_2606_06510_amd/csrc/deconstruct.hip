// Phase 1 of Alg. 1 (Ozaki II dense GEMM at phase level) on gfx950:
//   scan of the exponent spans (row/column maxima, T1 flags), 4-bit magnitude
//   codes for the max-magnitude pass, the power-of-two scales, and the
//   quantise -> centred residue -> E4M3 digit-plane split of Eq. (scale),
//   Eq. (modgemm), Eq. (sq-shortcut), Eq. (kar) and the carry-corrected
//   base-16 layout of the "e4m3 layout envelope" paragraph.
//
// All of it is HBM-bound streaming: A (column-major, rows strided) is read
// with lanes along the rows so every load instruction is a contiguous 512 B;
// B's columns are contiguous along k.  Outputs (codes, planes) are K-blocked
// byte planes [k/64][rows][64] (the GEMM's stage order), 16 bytes per lane.
#include "oz2_internal.h"

namespace {

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

__global__ void k_init(unsigned long long* rowbits, int mp, unsigned long long* colbits, int np,
                       uint32_t* Rmax, uint32_t* Kmax, int cslabs) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t nR = (size_t)cslabs * mp, nK = (size_t)cslabs * np;
  if (i < (size_t)mp) rowbits[i] = 0;
  if (i < (size_t)np) colbits[i] = 0;
  if (i < nR) Rmax[i] = 0;
  if (i < nK) Kmax[i] = 0;
}

// rows of a column-major matrix: lanes along the (contiguous) row index
__global__ void k_scan_rows(const double* __restrict__ A, int lda, int m, int k, int kchunk,
                            unsigned long long* rowbits) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  int l0 = blockIdx.y * kchunk;
  int l1 = min(k, l0 + kchunk);
  const double* p = A + i + (size_t)l0 * lda;
  unsigned long long mx = 0;
  int l = l0;
  for (; l + 4 <= l1; l += 4) {
    double x0 = p[0], x1 = p[(size_t)lda], x2 = p[2 * (size_t)lda], x3 = p[3 * (size_t)lda];
    mx = max(mx, max(max(abs_bits(x0), abs_bits(x1)), max(abs_bits(x2), abs_bits(x3))));
    p += 4 * (size_t)lda;
  }
  for (; l < l1; ++l, p += lda) mx = max(mx, abs_bits(*p));
  atomicMax(rowbits + i, mx);
}

// contiguous columns: one wave per column
__global__ void k_scan_cols(const double* __restrict__ B, int ldb, int n, int k,
                            unsigned long long* colbits) {
  int j = (int)((blockIdx.x * (size_t)blockDim.x + threadIdx.x) >> 6);
  int lane = threadIdx.x & 63;
  if (j >= n) return;
  const double* p = B + (size_t)j * ldb;
  unsigned long long mx = 0;
  for (int l = lane; l < k; l += 64) mx = max(mx, abs_bits(p[l]));
  for (int off = 32; off; off >>= 1) mx = max(mx, (unsigned long long)__shfl_xor((long long)mx, off));
  if (lane == 0) colbits[j] = mx;
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

// Row segment of 16 consecutive k for one row of A (TRANS) or column of B;
// a block of 256 threads covers 64 rows x 64 k.  A-side lanes run along the
// rows (each load instruction reads 512 contiguous bytes of a column of A);
// B-side lanes run along k (4 lanes read 512 contiguous bytes of a column
// of B).  The grid is one-dimensional: block b covers row block b % nrb and
// k block b / nrb (nrb = padded rows / 64).
template <bool TRANS>
__device__ __forceinline__ void seg_coords(int nrb, int& row, int& l0) {
  const int t = threadIdx.x;
  const int bx = (int)(blockIdx.x % (unsigned)nrb), by = (int)(blockIdx.x / (unsigned)nrb);
  if (TRANS) {
    row = bx * 64 + (t & 63);
    l0 = by * 64 + (t >> 6) * 16;
  } else {
    row = bx * 64 + (t >> 2);
    l0 = by * 64 + (t & 3) * 16;
  }
}

// byte offset of (row, k) in a K-blocked plane [kp/64][rows_pad][64]
__device__ __forceinline__ size_t kblocked(int row, int l, int rows_pad) {
  return ((size_t)(l >> 6) * rows_pad + row) * OZ2_KBLK + (l & 63);
}

template <bool TRANS>
__device__ __forceinline__ void load_seg(const double* __restrict__ X, int ld, int rows, int k,
                                         int row, int l0, bool zero, double (&x)[16]) {
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    int l = l0 + j;
    bool ok = !zero && row < rows && l < k;
    size_t off = TRANS ? ((size_t)row + (size_t)l * ld) : ((size_t)l + (size_t)row * ld);
    x[j] = ok ? X[off] : 0.0;
  }
}

template <bool TRANS>
__global__ void k_codes(const double* __restrict__ X, int ld, int rows, int nrb, int k, int kp,
                        const unsigned long long* __restrict__ bits, uint8_t* __restrict__ codes) {
  const int rows_pad = nrb * 64;
  int row, l0;
  seg_coords<TRANS>(nrb, row, l0);
  unsigned long long b = row < rows ? bits[row] : 0ull;
  bool t1 = b >= kInfBits;
  int E = (b == 0 || t1) ? 0 : exp_of_bits(b);
  double x[16];
  load_seg<TRANS>(X, ld, rows, k, row, l0, t1, x);
  uint32_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q)
    w[q] = pack4_fp8(code_of(x[4 * q], E), code_of(x[4 * q + 1], E), code_of(x[4 * q + 2], E),
                     code_of(x[4 * q + 3], E));
  uint4 v = make_uint4(w[0], w[1], w[2], w[3]);
  *reinterpret_cast<uint4*>(codes + kblocked(row, l0, rows_pad)) = v;
}

// widths sigma = min(62, c - ceil(ell(R)/2)), ell(x) = ceil(log2 x) (0 for x <= 1)
__device__ __forceinline__ int width_of(unsigned long long R, int budget) {
  int ell = (R > 1) ? (64 - __clzll((long long)(R - 1))) : 0;
  return min(62, budget - ((ell + 1) >> 1));
}

__global__ void k_scales(Oz2Dims d, const unsigned long long* __restrict__ rowbits,
                         const unsigned long long* __restrict__ colbits,
                         const uint32_t* __restrict__ Rmax, const uint32_t* __restrict__ Kmax,
                         int32_t* sA, int32_t* tB, uint32_t* fA, uint32_t* fB, int cA, int cB,
                         int* counters) {
  int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx == 0) { counters[0] = 0; counters[1] = 0; counters[2] = 0; counters[3] = 0; }
  bool fixed = (d.flags & 2u) != 0;   // OZ2_SCALE_FIXED
  unsigned long long fixedR = 256ull * (unsigned long long)d.k;
  if (idx < d.mp) {
    int i = idx;
    unsigned long long b = rowbits[i];
    int s = 0;
    uint32_t f = 0;
    if (i < d.m) {
      if (b >= kInfBits) {
        f = OZ2_T1;
      } else {
        int E = b ? exp_of_bits(b) : 0;
        unsigned long long R = fixedR;
        if (!fixed) {
          R = 0;
          for (int sl = 0; sl < d.cslabs; ++sl) R += Rmax[(size_t)sl * d.mp + i];
        }
        s = width_of(R, cA) - E;
      }
    }
    sA[i] = s;
    fA[i] = f;
  } else if (idx < d.mp + d.np) {
    int j = idx - d.mp;
    unsigned long long b = colbits[j];
    int t = 0;
    uint32_t f = 0;
    if (j < d.n) {
      if (b >= kInfBits) {
        f = OZ2_T1;
      } else {
        int E = b ? exp_of_bits(b) : 0;
        unsigned long long K = fixedR;
        if (!fixed) {
          K = 0;
          for (int sl = 0; sl < d.cslabs; ++sl) K += Kmax[(size_t)sl * d.np + j];
        }
        t = width_of(K, cB) - E;
      }
    }
    tB[j] = t;
    fB[j] = f;
  }
}

// Centred residue of the exact integer a (|a| <= 2^62, a double) modulo m:
// a = ah 2^32 + al (exact), t = ah (2^32 mod m) + al (exact, |t| < 2^42),
// r = t - m floor(t/m) with one correction each way (the fp64 quotient
// estimate of |t| < 2^42 is within 2^-18 of the true one).
__device__ __forceinline__ int centred_residue(double ah, double al, int m, int c32, double dinv) {
  double t = fma(ah, (double)c32, al);
  double q = floor(t * dinv);
  double r = fma(-q, (double)m, t);
  r = (r < 0.0) ? r + (double)m : r;
  r = (r >= (double)m) ? r - (double)m : r;
  int ri = (int)r;
  return (ri >= ((m + 1) >> 1)) ? ri - m : ri;
}

// Balanced base-s digits of a centred residue of m = s^2 (Eq. (sq-shortcut)):
// d0 = ((d + floor(s/2)) mod s) - floor(s/2), d1 = (d - d0)/s.
__device__ __forceinline__ void split_square(int dres, int s, int m, float inv_s, int& d0, int& d1) {
  int h = s >> 1;
  int u = dres + h + m;                  // in [0, 2m)
  int q = (int)((float)u * inv_s);
  int r = u - q * s;
  r += (r < 0) ? s : 0;
  r -= (r >= s) ? s : 0;
  d0 = r - h;
  d1 = (int)rintf((float)(dres - d0) * inv_s);
}

// Balanced base-16 digits with the carry correction of the "e4m3 layout
// envelope" paragraph: if d0+d1 is not E4M3-exact (odd and above 16 in
// magnitude), move one unit of base weight: (d0 - 16 sgn(d0), d1 + sgn(d0)).
__device__ __forceinline__ void split_tail(int dres, int& d0, int& d1) {
  d0 = ((dres + 8) & 15) - 8;
  d1 = (dres - d0) >> 4;
  int sm = d0 + d1;
  int am = sm < 0 ? -sm : sm;
  if (am > 16 && (am & 1)) {
    int sg = d0 > 0 ? 1 : -1;
    d0 -= 16 * sg;
    d1 += sg;
  }
}

template <bool TRANS>
__global__ void __launch_bounds__(256) k_split(Oz2Const c, const double* __restrict__ X, int ld,
                                               int rows, int rows_pad, int nrb, int k, int kp,
                                               const int32_t* __restrict__ scale,
                                               uint32_t* flags, uint8_t* __restrict__ planes,
                                               unsigned quant_tz) {
  int row, l0;
  seg_coords<TRANS>(nrb, row, l0);
  bool inrow = row < rows;
  uint32_t f = inrow ? flags[row] : 0u;
  int s = inrow ? scale[row] : 0;
  double x[16];
  load_seg<TRANS>(X, ld, rows, k, row, l0, (f & OZ2_T1) != 0, x);
  // quantise, Eq. (scale): exact (|a| <= 2^62 with at most 53 significant bits)
  double ah[16], al[16];
  bool t2 = false;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    double y = ldexp(x[j], s);
    double a = quant_tz ? trunc(y) : rint(y);
    t2 |= (x[j] != 0.0) && (a == 0.0);
    double h = floor(a * 0x1p-32);
    ah[j] = h;
    al[j] = fma(-h, 0x1p32, a);
  }
  if (t2) atomicOr(flags + row, OZ2_T2);
  const size_t pstride = (size_t)rows_pad * kp;
  uint8_t* base = planes + kblocked(row, l0, rows_pad);
  for (int i = 0; i < c.r; ++i) {
    const int m = c.m[i], c32 = c.c32[i], s_ = c.sq[i];
    const double dinv = c.dinv[i];
    float p0[16], p1[16], p2[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      int dres = centred_residue(ah[j], al[j], m, c32, dinv);
      int d0, d1;
      if (s_) split_square(dres, s_, m, c.finv_s[i], d0, d1);
      else split_tail(dres, d0, d1);
      p0[j] = (float)d0;
      p1[j] = (float)d1;
      p2[j] = (float)(d0 + d1);
    }
    uint8_t* dst = base + (size_t)c.pbase[i] * pstride;
    uint4 v0, v1;
    v0.x = pack4_fp8(p0[0], p0[1], p0[2], p0[3]);
    v0.y = pack4_fp8(p0[4], p0[5], p0[6], p0[7]);
    v0.z = pack4_fp8(p0[8], p0[9], p0[10], p0[11]);
    v0.w = pack4_fp8(p0[12], p0[13], p0[14], p0[15]);
    v1.x = pack4_fp8(p1[0], p1[1], p1[2], p1[3]);
    v1.y = pack4_fp8(p1[4], p1[5], p1[6], p1[7]);
    v1.z = pack4_fp8(p1[8], p1[9], p1[10], p1[11]);
    v1.w = pack4_fp8(p1[12], p1[13], p1[14], p1[15]);
    *reinterpret_cast<uint4*>(dst) = v0;
    *reinterpret_cast<uint4*>(dst + pstride) = v1;
    if (!s_) {
      uint4 v2;
      v2.x = pack4_fp8(p2[0], p2[1], p2[2], p2[3]);
      v2.y = pack4_fp8(p2[4], p2[5], p2[6], p2[7]);
      v2.z = pack4_fp8(p2[8], p2[9], p2[10], p2[11]);
      v2.w = pack4_fp8(p2[12], p2[13], p2[14], p2[15]);
      *reinterpret_cast<uint4*>(dst + 2 * pstride) = v2;
    }
  }
}

}  // namespace

hipError_t oz2_launch_init(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, hipStream_t s) {
  size_t n = (size_t)d.cslabs * (size_t)(d.mp > d.np ? d.mp : d.np);
  if ((size_t)d.mp > n) n = d.mp;
  if ((size_t)d.np > n) n = d.np;
  unsigned blocks = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(k_init, dim3(blocks), dim3(256), 0, s,
                     (unsigned long long*)(ws + L.rowbits), d.mp,
                     (unsigned long long*)(ws + L.colbits), d.np, (uint32_t*)(ws + L.Rmax),
                     (uint32_t*)(ws + L.Kmax), d.cslabs);
  return hipGetLastError();
}

hipError_t oz2_launch_scan(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, const double* A,
                           int lda, const double* B, int ldb, hipStream_t s) {
  int kchunk = 256;
  while ((d.k + kchunk - 1) / kchunk > 16384) kchunk *= 2;   // keep grid.y small
  dim3 ga((d.m + 255) / 256, (d.k + kchunk - 1) / kchunk);
  hipLaunchKernelGGL(k_scan_rows, ga, dim3(256), 0, s, A, lda, d.m, d.k, kchunk,
                     (unsigned long long*)(ws + L.rowbits));
  dim3 gb((d.n + 3) / 4);
  hipLaunchKernelGGL(k_scan_cols, gb, dim3(256), 0, s, B, ldb, d.n, d.k,
                     (unsigned long long*)(ws + L.colbits));
  return hipGetLastError();
}

hipError_t oz2_launch_codes(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, const double* A,
                            int lda, const double* B, int ldb, hipStream_t s) {
  dim3 ga((d.mp / 64) * (d.kp / 64));
  hipLaunchKernelGGL(k_codes<true>, ga, dim3(256), 0, s, A, lda, d.m, d.mp / 64, d.k, d.kp,
                     (const unsigned long long*)(ws + L.rowbits), ws + L.codesA);
  dim3 gb((d.np / 64) * (d.kp / 64));
  hipLaunchKernelGGL(k_codes<false>, gb, dim3(256), 0, s, B, ldb, d.n, d.np / 64, d.k, d.kp,
                     (const unsigned long long*)(ws + L.colbits), ws + L.codesB);
  return hipGetLastError();
}

hipError_t oz2_launch_scales(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                             uint8_t* ws, hipStream_t s) {
  unsigned blocks = (unsigned)((d.mp + d.np + 255) / 256);
  hipLaunchKernelGGL(k_scales, dim3(blocks), dim3(256), 0, s, d,
                     (const unsigned long long*)(ws + L.rowbits),
                     (const unsigned long long*)(ws + L.colbits), (const uint32_t*)(ws + L.Rmax),
                     (const uint32_t*)(ws + L.Kmax), (int32_t*)(ws + L.sA), (int32_t*)(ws + L.tB),
                     (uint32_t*)(ws + L.flagsA), (uint32_t*)(ws + L.flagsB), c.cA, c.cB,
                     (int*)(ws + L.counters));
  return hipGetLastError();
}

hipError_t oz2_launch_split(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                            const double* A, int lda, const double* B, int ldb, hipStream_t s) {
  unsigned tz = (d.flags & 4u) ? 1u : 0u;   // OZ2_QUANT_TZ
  dim3 ga((d.mp / 64) * (d.kp / 64));
  hipLaunchKernelGGL(k_split<true>, ga, dim3(256), 0, s, c, A, lda, d.m, d.mp, d.mp / 64, d.k,
                     d.kp, (const int32_t*)(ws + L.sA), (uint32_t*)(ws + L.flagsA),
                     ws + L.planesA, tz);
  dim3 gb((d.np / 64) * (d.kp / 64));
  hipLaunchKernelGGL(k_split<false>, gb, dim3(256), 0, s, c, B, ldb, d.n, d.np, d.np / 64, d.k,
                     d.kp, (const int32_t*)(ws + L.tB), (uint32_t*)(ws + L.flagsB),
                     ws + L.planesB, tz);
  return hipGetLastError();
}
