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
#include <mutex>

#include "oz2_device.h"

namespace {

// zero the row (side A) / column (side B) maxima the scans and the code GEMM
// accumulate with atomics, and the operand's fallback-list count (the list
// is filled by k_scales (T1) and k_split (T2) of this deconstruction)
__global__ void k_init(unsigned long long* rowbits, int mp, unsigned long long* colbits, int np,
                       uint32_t* Rmax, uint32_t* Kmax, int cslabs, int* counters, int side) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t nR = (size_t)cslabs * mp, nK = (size_t)cslabs * np;
  if (side & OZ2_SIDE_A) {
    if (i < (size_t)mp) rowbits[i] = 0;
    if (i < nR) Rmax[i] = 0;
    if (i == 0) counters[0] = 0;
  }
  if (side & OZ2_SIDE_B) {
    if (i < (size_t)np) colbits[i] = 0;
    if (i < nK) Kmax[i] = 0;
    if (i == 0) counters[1] = 0;
  }
}

// rows of a column-major matrix: lanes along the (contiguous) row index, two
// rows per thread (16-byte loads when the caller has checked the alignment),
// eight loads in flight; one k-chunk per grid row, combined with atomicMax.
__global__ void __launch_bounds__(256) k_scan_rows(const double* __restrict__ A, int lda, int m, int k,
                                                   int kchunk, unsigned vec,
                                                   unsigned long long* rowbits) {
  const int i = 2 * (blockIdx.x * blockDim.x + threadIdx.x);
  if (i >= m) return;
  const int l0 = blockIdx.y * kchunk;
  const int l1 = min(k, l0 + kchunk);
  const bool pair = vec && i + 1 < m;
  unsigned long long m0 = 0, m1 = 0;
  int l = l0;
  if (pair) {
    const double* p = A + i + (size_t)l0 * lda;
    for (; l + 8 <= l1; l += 8) {
      double2 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = *reinterpret_cast<const double2*>(p + (size_t)u * lda);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        m0 = max(m0, abs_bits(v[u].x));
        m1 = max(m1, abs_bits(v[u].y));
      }
      p += 8 * (size_t)lda;
    }
  }
  for (; l < l1; ++l) {
    const double* p = A + i + (size_t)l * lda;
    m0 = max(m0, abs_bits(p[0]));
    if (i + 1 < m) m1 = max(m1, abs_bits(p[1]));
  }
  atomicMax(rowbits + i, m0);
  if (i + 1 < m) atomicMax(rowbits + i + 1, m1);
}

// contiguous columns: one wave per column, 16-byte loads (1 KiB per wave
// instruction), four in flight per lane
__global__ void __launch_bounds__(256) k_scan_cols(const double* __restrict__ B, int ldb, int n, int k,
                                                   unsigned vec, unsigned long long* colbits) {
  int j = (int)((blockIdx.x * (size_t)blockDim.x + threadIdx.x) >> 6);
  int lane = threadIdx.x & 63;
  if (j >= n) return;
  const double* p = B + (size_t)j * ldb;
  unsigned long long mx = 0;
  int l = 0;
  if (vec) {
    for (; l + 512 <= k; l += 512) {
      double2 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const double2*>(p + l + 128 * u + 2 * lane);
#pragma unroll
      for (int u = 0; u < 4; ++u) mx = max(mx, max(abs_bits(v[u].x), abs_bits(v[u].y)));
    }
  }
  for (l += lane; l < k; l += 64) mx = max(mx, abs_bits(p[l]));
  for (int off = 32; off; off >>= 1) mx = max(mx, (unsigned long long)__shfl_xor((long long)mx, off));
  if (lane == 0) colbits[j] = mx;
}

// Row segment of 16 consecutive k for one row of A (TRANS) or column of B.
// A tile of 256 threads covers 64 rows x 64 k (one K-block): thread t owns
// row t/4, k chunk t%4, so every 16-byte store of a wave fills 1 KiB of
// contiguous K-blocked plane; A's loads read 4 x 128 B per instruction, B's
// 4 lanes read 512 contiguous bytes of a column.  Tile tl of a 1-D sequence
// covers row block tl % nrb and k block tl / nrb (nrb = padded rows / 64).
__device__ __forceinline__ void seg_coords(int tl, int nrb, int& row, int& l0) {
  const int t = threadIdx.x;
  const int bx = tl % nrb, by = tl / nrb;
  row = bx * 64 + (t >> 2);
  l0 = by * 64 + (t & 3) * 16;
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

// As load_seg; a full 16-element segment of a contiguous column (B side) is
// read with 16-byte loads when the caller has checked X and ld for alignment.
template <bool TRANS>
__device__ __forceinline__ void load_seg_fast(const double* __restrict__ X, int ld, int rows, int k,
                                              int row, int l0, bool zero, bool vec,
                                              double (&x)[16]) {
  if (!TRANS && vec && !zero && row < rows && l0 + 16 <= k) {
    const double2* p = reinterpret_cast<const double2*>(X + (size_t)row * ld + l0);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const double2 v = p[j];
      x[2 * j] = v.x;
      x[2 * j + 1] = v.y;
    }
  } else {
    load_seg<TRANS>(X, ld, rows, k, row, l0, zero, x);
  }
}

// Contiguous-column operand (B): a tile of 64 columns x 64 k is read with
// coalesced 16-byte loads (32 lanes per 512-byte column segment) into LDS, and
// each thread then takes its 16 consecutive k of column t/4 (the layout the
// plane stores need).  The caller synchronises before the tile is reused.
constexpr int TPITCH = 66;   // doubles per staged column: 16-byte aligned, banks spread

__device__ __forceinline__ void stage_cols(const double* __restrict__ X, int ld, int rows, int k,
                                           int row0, int l00, bool vec, double* tile) {
  const int t = threadIdx.x;
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int idx = it * 256 + t;
    const int c = idx >> 5, kk = (idx & 31) << 1;
    const int r = row0 + c, l = l00 + kk;
    double2 v = make_double2(0.0, 0.0);
    if (r < rows) {
      const double* p = X + (size_t)r * ld + l;
      if (vec && l + 1 < k) {
        v = *reinterpret_cast<const double2*>(p);
      } else {
        if (l < k) v.x = p[0];
        if (l + 1 < k) v.y = p[1];
      }
    }
    *reinterpret_cast<double2*>(tile + c * TPITCH + kk) = v;
  }
}

__device__ __forceinline__ void take_cols(const double* tile, bool zero, double (&x)[16]) {
  const int t = threadIdx.x;
  const double* p = tile + (t >> 2) * TPITCH + (t & 3) * 16;
#pragma unroll
  for (int j = 0; j < 16; j += 2) {
    const double2 v = *reinterpret_cast<const double2*>(p + j);
    x[j] = zero ? 0.0 : v.x;
    x[j + 1] = zero ? 0.0 : v.y;
  }
}

// Codes for the max-magnitude pass, in two steps so that each operand's FP64
// input is read once here (the scan and the codes share the read):
//
// 1. k_scan_codes_rows / _cols (one 64x64 tile of 64 rows or columns x 64 k
//    per workgroup): the tile-row maxima of |x| (folded into the row maxima
//    with atomicMax), their frexp exponents Et (int16 [k/64][rows]), and per
//    element a byte relative to Et, stored in the K-blocked codes layout:
//      bit 7: x != 0;  bits 4..6: min(Et - e, 4);  bit 3: sticky;
//      bits 0..2: floor(16 f) - 8,   where |x| = f 2^e, f in [1/2, 1),
//    the sticky bit telling whether 16 f has bits below its integer part.
// 2. k_rebase (both operands, one launch, in place): with E the exponent of
//    the whole row's maximum and d = min(E - Et + (E_t - e), 4) = min(E - e, 4),
//    the code ceil(16 |x| 2^-E) = ceil((q + rho) 2^-d), q = floor(16 f) in
//    [8, 15], rho in [0, 1), is q + sticky for d = 0, 1 for d >= 4 (x != 0),
//    else floor(q / 2^d) + 1 if q mod 2^d or sticky is nonzero, q / 2^d if not:
//    exactly the code of code_of(), from the byte alone (the three cases are
//    (q + 2^d - 1 + sticky) >> d).  T1 rows (a NaN or Inf entry) get codes 0,
//    as before.
__device__ __forceinline__ uint32_t local_code(unsigned long long b, int Et) {
  uint32_t hi = (uint32_t)(b >> 32);
  const uint32_t lo = (uint32_t)b;
  // normal x: every field from the high word and one test of the low one
  uint32_t q3 = (hi >> 17) & 7u;                          // floor(16 f) - 8
  uint32_t st = ((hi & 0x1FFFFu) | lo) ? 8u : 0u;         // bits of 16 f below 1
  int e = (int)(hi >> 20) - 1022;
  if ((hi >> 20) == 0u) {   // zero or subnormal (rare): normalise the mantissa
    if ((hi | lo) == 0u) return 0u;
    const int z = __clzll((long long)b);                  // >= 12
    const unsigned long long man = (b << (z - 11)) & 0xFFFFFFFFFFFFFull;
    q3 = (uint32_t)(man >> 49);
    st = (man & 0x1FFFFFFFFFFFFull) ? 8u : 0u;
    e = (64 - z) - 1074;
  }
  const int dt = min(Et - e, 4);
  return 0x80u | ((uint32_t)dt << 4) | st | q3;
}

// Rows of A (contiguous along the row index): thread t reads rows 2(t%32),
// 2(t%32)+1 of k = t/32 + 8j (j < 8) with 16-byte loads (each wave
// instruction covers 512 contiguous bytes of two columns); the 64 x 64 bytes
// are transposed through LDS so that each thread stores 16 consecutive k of
// one row.
__global__ void __launch_bounds__(256) k_scan_codes_rows(const double* __restrict__ X, int ld,
                                                         int rows, int nrb, int k, unsigned vec,
                                                         unsigned long long* bits, int16_t* et,
                                                         uint8_t* __restrict__ codes) {
  __shared__ __attribute__((aligned(16))) uint8_t T[64][80];
  __shared__ unsigned long long mx[8][64];
  const int rows_pad = nrb * 64;
  const int t = threadIdx.x;
  const int bx = (int)(blockIdx.x % (unsigned)nrb), by = (int)(blockIdx.x / (unsigned)nrb);
  const int p = t & 31, g = t >> 5;
  const int r0 = bx * 64 + 2 * p, lbase = by * 64;
  double2 v[8];
  if (vec && bx * 64 + 64 <= rows && lbase + 64 <= k) {   // interior tile (uniform)
    const double* q = X + (size_t)(lbase + g) * ld + r0;
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const double2*>(q + (size_t)(8 * j) * ld);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int l = lbase + g + 8 * j;
      v[j] = make_double2(0.0, 0.0);
      if (l < k) {
        const double* q = X + (size_t)l * ld + r0;
        if (vec && r0 + 1 < rows) {
          v[j] = *reinterpret_cast<const double2*>(q);
        } else {
          if (r0 < rows) v[j].x = q[0];
          if (r0 + 1 < rows) v[j].y = q[1];
        }
      }
    }
  }
  unsigned long long m0 = 0, m1 = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    m0 = max(m0, abs_bits(v[j].x));
    m1 = max(m1, abs_bits(v[j].y));
  }
  mx[g][2 * p] = m0;
  mx[g][2 * p + 1] = m1;
  __syncthreads();
  if (t < 64) {
    unsigned long long m = mx[0][t];
#pragma unroll
    for (int u = 1; u < 8; ++u) m = max(m, mx[u][t]);
    const int row = bx * 64 + t;
    if (row < rows && m) atomicMax(bits + row, m);
    et[(size_t)by * rows_pad + row] = (int16_t)(m ? exp_of_bits(m) : 0);
    mx[0][t] = m;   // only thread t reads column t of mx
  }
  __syncthreads();
  const unsigned long long t0 = mx[0][2 * p], t1 = mx[0][2 * p + 1];
  const int E0 = t0 ? exp_of_bits(t0) : 0, E1 = t1 ? exp_of_bits(t1) : 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int c = g + 8 * j;
    T[2 * p][c] = (uint8_t)local_code(abs_bits(v[j].x), E0);
    T[2 * p + 1][c] = (uint8_t)local_code(abs_bits(v[j].y), E1);
  }
  __syncthreads();
  const int row = bx * 64 + (t >> 2), l0 = lbase + (t & 3) * 16;
  const uint4 o = *reinterpret_cast<const uint4*>(&T[t >> 2][(t & 3) * 16]);
  *reinterpret_cast<uint4*>(codes + kblocked(row, l0, rows_pad)) = o;
}

// Columns of B (contiguous along k): thread t reads k 2(t%32), 2(t%32)+1 of
// columns t/32 + 8j with 16-byte loads (512 contiguous bytes of one column per
// half-wave instruction); a column's tile maximum is a max-reduction over the
// 32 lanes of a half-wave; the bytes are transposed through LDS as for A.
__global__ void __launch_bounds__(256) k_scan_codes_cols(const double* __restrict__ X, int ld,
                                                         int rows, int nrb, int k, unsigned vec,
                                                         unsigned long long* bits, int16_t* et,
                                                         uint8_t* __restrict__ codes) {
  __shared__ __attribute__((aligned(16))) uint8_t T[64][80];
  const int rows_pad = nrb * 64;
  const int t = threadIdx.x;
  // k-blocks fastest: consecutive workgroups read consecutive 512-byte pieces
  // of the same 64 columns (DRAM pages are filled in order)
  const int nkb = (int)(gridDim.x / (unsigned)nrb);
  const int by = (int)(blockIdx.x % (unsigned)nkb), bx = (int)(blockIdx.x / (unsigned)nkb);
  const int p = t & 31, kk = 2 * p, g = t >> 5;
  const int l = by * 64 + kk;
  double2 v[8];
  if (vec && bx * 64 + 64 <= rows && by * 64 + 64 <= k) {   // interior tile (uniform)
    const double* q = X + (size_t)(bx * 64 + g) * ld + l;
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const double2*>(q + (size_t)(8 * j) * ld);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int col = bx * 64 + g + 8 * j;
      v[j] = make_double2(0.0, 0.0);
      if (col < rows) {
        const double* q = X + (size_t)col * ld + l;
        if (vec && l + 1 < k) {
          v[j] = *reinterpret_cast<const double2*>(q);
        } else {
          if (l < k) v[j].x = q[0];
          if (l + 1 < k) v[j].y = q[1];
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int cc = g + 8 * j, col = bx * 64 + cc;
    const unsigned long long a0 = abs_bits(v[j].x), a1 = abs_bits(v[j].y);
    unsigned long long m = max(a0, a1);
#pragma unroll
    for (int off = 16; off; off >>= 1)
      m = max(m, (unsigned long long)__shfl_xor((long long)m, off, 32));
    if (p == 0) {
      if (col < rows && m) atomicMax(bits + col, m);
      et[(size_t)by * rows_pad + col] = (int16_t)(m ? exp_of_bits(m) : 0);
    }
    const int E = m ? exp_of_bits(m) : 0;
    const uint32_t w = local_code(a0, E) | (local_code(a1, E) << 8);
    *reinterpret_cast<uint16_t*>(&T[cc][kk]) = (uint16_t)w;
  }
  __syncthreads();
  const int row = bx * 64 + (t >> 2), l0 = by * 64 + (t & 3) * 16;
  const uint4 o = *reinterpret_cast<const uint4*>(&T[t >> 2][(t & 3) * 16]);
  *reinterpret_cast<uint4*>(codes + kblocked(row, l0, rows_pad)) = o;
}

// code of one byte of step 1 given D = E - Et: with d = min(D + dt, 4), the
// ceiling above is (q + 2^d - 1 + sticky) >> d for every d in [0, 4]
__device__ __forceinline__ float rebase_code(uint32_t y, int D) {
  const int d = min(D + (int)((y >> 4) & 7u), 4);
  const int c = (7 + (int)(y & 7u) + (int)((y >> 3) & 1u) + (1 << d)) >> d;
  return (y & 0x80u) ? (float)c : 0.0f;
}

// Step 2 for both operands, in place: one thread per 64-byte row segment of
// one k-block (threads [0, nA) on A, then B), four 16-byte loads in flight.
// Since d = min(D + dt, 4) depends on D only through min(D, 4), the E4M3 code
// of every byte for every D is a 5 x 256-byte table, built per workgroup in
// LDS; a byte then costs a shift, an add and one LDS byte read.
__global__ void __launch_bounds__(256) k_rebase(uint8_t* codesA, const int16_t* __restrict__ etA,
                                                const unsigned long long* __restrict__ bitsA,
                                                int mp, size_t nA, uint8_t* codesB,
                                                const int16_t* __restrict__ etB,
                                                const unsigned long long* __restrict__ bitsB,
                                                int np, size_t nB) {
  __shared__ uint8_t lut[5 * 256];
  for (int e = threadIdx.x; e < 5 * 256; e += blockDim.x)
    lut[e] = (uint8_t)(__builtin_amdgcn_cvt_pk_fp8_f32(rebase_code((uint32_t)(e & 255), e >> 8),
                                                       0.0f, 0, false) & 0xFF);
  __syncthreads();
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint8_t* codes = codesA;
  const int16_t* et = etA;
  const unsigned long long* bits = bitsA;
  int rp = mp;
  if (i >= nA) {
    i -= nA;
    if (i >= nB) return;
    codes = codesB;
    et = etB;
    bits = bitsB;
    rp = np;
  }
  // segment i = (k-block, row): et is [k/64][rows], the codes [k/64][rows][64];
  // every load first (one round of latency), then the lookups
  const int row = (int)(i % (size_t)rp);
  uint4* q = reinterpret_cast<uint4*>(codes) + 4 * i;
  uint4 y[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) y[u] = q[u];
  const unsigned long long b = bits[row];
  const int et_i = (int)et[i];
  if (b == 0 || b >= kInfBits) {   // all-zero row, or T1: codes 0
#pragma unroll
    for (int u = 0; u < 4; ++u) q[u] = make_uint4(0u, 0u, 0u, 0u);
    return;
  }
  const uint8_t* t = lut + 256 * min(exp_of_bits(b) - et_i, 4);
  auto word = [t](uint32_t w) {
    return (uint32_t)t[w & 0xFFu] | ((uint32_t)t[(w >> 8) & 0xFFu] << 8) |
           ((uint32_t)t[(w >> 16) & 0xFFu] << 16) | ((uint32_t)t[w >> 24] << 24);
  };
#pragma unroll
  for (int u = 0; u < 4; ++u)
    q[u] = make_uint4(word(y[u].x), word(y[u].y), word(y[u].z), word(y[u].w));
}

__global__ void k_scales(Oz2Dims d, const unsigned long long* __restrict__ rowbits,
                         const unsigned long long* __restrict__ colbits,
                         const uint32_t* __restrict__ Rmax, const uint32_t* __restrict__ Kmax,
                         int32_t* sA, int32_t* tB, int32_t* eA, int32_t* eB, uint32_t* fA,
                         uint32_t* fB, int cA, int cB, int* counters, int* listA, int* listB,
                         int side) {
  int idx = blockIdx.x * blockDim.x + threadIdx.x;
  bool fixed = (d.flags & 2u) != 0;   // OZ2_SCALE_FIXED
  const bool force = (d.flags & 16u) != 0;   // OZ2_FORCE_FALLBACK: every row of A natively
  unsigned long long fixedR = 256ull * (unsigned long long)d.k;
  if (idx < d.mp) {
    if (!(side & OZ2_SIDE_A)) return;
    int i = idx;
    unsigned long long b = rowbits[i];
    int s = 0, E = 0;
    uint32_t f = 0;
    if (i < d.m) {
      if (b >= kInfBits) {
        f = OZ2_T1;
      } else {
        E = b ? exp_of_bits(b) : 0;
        unsigned long long R = fixedR;
        if (!fixed) {
          R = 0;
          for (int sl = 0; sl < d.cslabs; ++sl) R += Rmax[(size_t)sl * d.mp + i];
        }
        s = width_of(R, cA) - E;
      }
    }
    sA[i] = s;
    eA[i] = E;
    fA[i] = f;
    if (i < d.m && (force || f)) listA[atomicAdd(counters + 0, 1)] = i;
  } else if (idx < d.mp + d.np) {
    if (!(side & OZ2_SIDE_B)) return;
    int j = idx - d.mp;
    unsigned long long b = colbits[j];
    int t = 0, E = 0;
    uint32_t f = 0;
    if (j < d.n) {
      if (b >= kInfBits) {
        f = OZ2_T1;
      } else {
        E = b ? exp_of_bits(b) : 0;
        unsigned long long K = fixedR;
        if (!fixed) {
          K = 0;
          for (int sl = 0; sl < d.cslabs; ++sl) K += Kmax[(size_t)sl * d.np + j];
        }
        t = width_of(K, cB) - E;
      }
    }
    tB[j] = t;
    eB[j] = E;
    fB[j] = f;
    if (j < d.n && !force && f) listB[atomicAdd(counters + 1, 1)] = j;
  }
}

// residue -> plane bytes: entry toff[i] + d = E4M3(d0) | E4M3(d1) << 8 |
// E4M3(d0 + d1) << 16 | E4M3(-16 d1) << 24 (exact: |16 d1| <= 256; the
// last two bytes are used for nonsquare moduli only, the fourth by the
// single-launch batched kernel)
__global__ void k_plane_tables(Oz2Const c, uint32_t* tab) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= c.tabsz) return;
  int i = 0;
  while (i + 1 < c.r && idx >= c.toff[i + 1] - c.m[i + 1] / 2) ++i;
  const int m = c.m[i];
  const int d = idx - c.toff[i];
  int d0, d1;
  oz2_digits(d, m, c.sq[i], d0, d1);
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32((float)d0, (float)d1, 0, false);
  const int hi = __builtin_amdgcn_cvt_pk_fp8_f32((float)(d0 + d1), 0.0f, 0, false);
  const int b3 = __builtin_amdgcn_cvt_pk_fp8_f32((float)(-16 * d1), 0.0f, 0, false);
  tab[idx] = ((uint32_t)lo & 0xFFFFu) | (((uint32_t)hi & 0xFFu) << 16) |
             (((uint32_t)b3 & 0xFFu) << 24);
}

// Plane bytes are written once and read back only by the residue GEMMs, after
// the other operand's split: non-temporal stores keep them from displacing
// that operand's FP64 input in the caches while it waits to be re-read.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store_stream(uint8_t* p, uint4 v) {
  __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4*>(p));
}

// One operand of the split: where its FP64 input, scales, flags, planes and
// fallback list are, and its 64x64 tile count.
struct SplitSide {
  const double* X;
  int ld, rows, rows_pad, nrb, ntiles;
  const int32_t* scale;
  uint32_t* flags;
  uint8_t* planes;
  unsigned vec;
  int* count;
  int* list;
  int listed;          // every row is on the fallback list already (FORCE_FALLBACK on A)
};

// Quantise (Eq. (scale)) and split into E4M3 digit planes one 64x64 tile
// (64 rows x 64 k) of one operand.
template <bool TRANS>
__device__ __forceinline__ void split_tile(const Oz2Const& c, const SplitSide& S, int tl, int k,
                                           int kp, const uint32_t* tab, unsigned quant_tz) {
  const size_t pstride = (size_t)S.rows_pad * kp;
  int row, l0;
  seg_coords(tl, S.nrb, row, l0);
  const bool inrow = row < S.rows;
  const uint32_t f = inrow ? S.flags[row] : 0u;
  const int sc = inrow ? S.scale[row] : 0;
  double x[16];
  load_seg_fast<TRANS>(S.X, S.ld, S.rows, k, row, l0, (f & OZ2_T1) != 0, S.vec != 0, x);
  // quantise: exact (|a| <= 2^62 with at most 53 significant bits)
  double ah[16], al[16];
  bool t2 = false;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const double y = ldexp(x[j], sc);
    const double a = quant_tz ? trunc(y) : rint(y);
    t2 |= (x[j] != 0.0) && (a == 0.0);
    const double h = floor(a * 0x1p-32);
    ah[j] = h;
    al[j] = fma(-h, 0x1p32, a);
  }
  // the first tile to flag a row adds it to the fallback list (unless every
  // row is listed already)
  if (t2 && !(atomicOr(S.flags + row, OZ2_T2) & (OZ2_T1 | OZ2_T2)) && !S.listed)
    S.list[atomicAdd(S.count, 1)] = row;
  uint8_t* base = S.planes + kblocked(row, l0, S.rows_pad);
  for (int i = 0; i < c.r; ++i) {
    const double m = (double)c.m[i], c32 = (double)c.c32[i], dinv = c.dinv[i];
    const int to = c.toff[i];
    uint32_t e[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) e[j] = tab[to + centred_residue(ah[j], al[j], m, c32, dinv)];
    uint8_t* dst = base + (size_t)c.pbase[i] * pstride;
    uint4 v0, v1;
    v0.x = gather_byte(e[0], e[1], e[2], e[3], 0x05010400u);
    v0.y = gather_byte(e[4], e[5], e[6], e[7], 0x05010400u);
    v0.z = gather_byte(e[8], e[9], e[10], e[11], 0x05010400u);
    v0.w = gather_byte(e[12], e[13], e[14], e[15], 0x05010400u);
    v1.x = gather_byte(e[0], e[1], e[2], e[3], 0x05010501u);
    v1.y = gather_byte(e[4], e[5], e[6], e[7], 0x05010501u);
    v1.z = gather_byte(e[8], e[9], e[10], e[11], 0x05010501u);
    v1.w = gather_byte(e[12], e[13], e[14], e[15], 0x05010501u);
    store_stream(dst, v0);
    store_stream(dst + pstride, v1);
    if (!c.sq[i]) {
      uint4 v2;
      v2.x = gather_byte(e[0], e[1], e[2], e[3], 0x05010602u);
      v2.y = gather_byte(e[4], e[5], e[6], e[7], 0x05010602u);
      v2.z = gather_byte(e[8], e[9], e[10], e[11], 0x05010602u);
      v2.w = gather_byte(e[12], e[13], e[14], e[15], 0x05010602u);
      store_stream(dst + 2 * pstride, v2);
    }
  }
}

// The split of both operands in one persistent-style launch (no drain between
// them): B's tiles first, while B is still in the memory-side cache after its
// codes pass, then A's (measured at 4096^3: 402 us for the deconstruction,
// against 417 with the tiles of A and B interleaved and 420 with A first).
// Each workgroup first copies the residue->bytes tables (sum of the moduli
// entries, <= 42 KiB) into LDS.
__global__ void __launch_bounds__(256) k_split(Oz2Const c, SplitSide SA, SplitSide SB, int k,
                                               int kp, const uint32_t* __restrict__ gtab,
                                               unsigned quant_tz) {
  extern __shared__ __attribute__((aligned(16))) uint32_t tab[];
  for (int i = threadIdx.x; i < c.tabsz; i += blockDim.x) tab[i] = gtab[i];
  __syncthreads();
  const int total = SA.ntiles + SB.ntiles;
  for (int t = blockIdx.x; t < total; t += gridDim.x) {
    const int side = t < SB.ntiles ? 1 : 0;
    const int tl = side ? t : t - SB.ntiles;
    if (side == 0) split_tile<true>(c, SA, tl, k, kp, tab, quant_tz);
    else split_tile<false>(c, SB, tl, k, kp, tab, quant_tz);
  }
}

}  // namespace

hipError_t oz2_launch_init(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, int side,
                           hipStream_t s) {
  size_t n = (size_t)d.cslabs * (size_t)(d.mp > d.np ? d.mp : d.np);
  if ((size_t)d.mp > n) n = d.mp;
  if ((size_t)d.np > n) n = d.np;
  unsigned blocks = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(k_init, dim3(blocks), dim3(256), 0, s,
                     (unsigned long long*)(ws + L.rowbits), d.mp,
                     (unsigned long long*)(ws + L.colbits), d.np, (uint32_t*)(ws + L.Rmax),
                     (uint32_t*)(ws + L.Kmax), d.cslabs, (int*)(ws + L.counters), side);
  return hipGetLastError();
}

hipError_t oz2_launch_scan(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, const double* A,
                           int lda, const double* B, int ldb, int side, hipStream_t s) {
  if (side & OZ2_SIDE_A) {
    // rows: 512 per workgroup; k chunks sized for >= ~2048 workgroups when k allows
    const int gx = (d.m + 511) / 512;
    int kchunk = 32;
    while ((long long)gx * ((d.k + kchunk - 1) / kchunk) > 4096 && kchunk < 4096) kchunk *= 2;
    while ((d.k + kchunk - 1) / kchunk > 65535) kchunk *= 2;
    const unsigned vecA = ((uintptr_t)A % 16 == 0 && lda % 2 == 0) ? 1u : 0u;
    dim3 ga(gx, (d.k + kchunk - 1) / kchunk);
    hipLaunchKernelGGL(k_scan_rows, ga, dim3(256), 0, s, A, lda, d.m, d.k, kchunk, vecA,
                       (unsigned long long*)(ws + L.rowbits));
  }
  if (side & OZ2_SIDE_B) {
    dim3 gb((d.n + 3) / 4);
    const unsigned vecB = ((uintptr_t)B % 16 == 0 && ldb % 2 == 0) ? 1u : 0u;
    hipLaunchKernelGGL(k_scan_cols, gb, dim3(256), 0, s, B, ldb, d.n, d.k, vecB,
                       (unsigned long long*)(ws + L.colbits));
  }
  return hipGetLastError();
}

hipError_t oz2_launch_scan_codes(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws,
                                 const double* A, int lda, const double* B, int ldb, int side,
                                 hipStream_t s) {
  if (side & OZ2_SIDE_A) {
    dim3 ga((d.mp / 64) * (d.kp / 64));
    const unsigned vecA = ((uintptr_t)A % 16 == 0 && lda % 2 == 0) ? 1u : 0u;
    hipLaunchKernelGGL(k_scan_codes_rows, ga, dim3(256), 0, s, A, lda, d.m, d.mp / 64, d.k, vecA,
                       (unsigned long long*)(ws + L.rowbits), (int16_t*)(ws + L.etA),
                       ws + L.codesA);
  }
  if (side & OZ2_SIDE_B) {
    dim3 gb((d.np / 64) * (d.kp / 64));
    const unsigned vecB = ((uintptr_t)B % 16 == 0 && ldb % 2 == 0) ? 1u : 0u;
    hipLaunchKernelGGL(k_scan_codes_cols, gb, dim3(256), 0, s, B, ldb, d.n, d.np / 64, d.k, vecB,
                       (unsigned long long*)(ws + L.colbits), (int16_t*)(ws + L.etB),
                       ws + L.codesB);
  }
  return hipGetLastError();
}

hipError_t oz2_launch_rebase(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, int side,
                             hipStream_t s) {
  const size_t nA = (side & OZ2_SIDE_A) ? (size_t)d.mp * (d.kp / 64) : 0;
  const size_t nB = (side & OZ2_SIDE_B) ? (size_t)d.np * (d.kp / 64) : 0;
  if (nA + nB == 0) return hipSuccess;
  hipLaunchKernelGGL(k_rebase, dim3((unsigned)((nA + nB + 255) / 256)), dim3(256), 0, s,
                     ws + L.codesA, (const int16_t*)(ws + L.etA),
                     (const unsigned long long*)(ws + L.rowbits), d.mp, nA, ws + L.codesB,
                     (const int16_t*)(ws + L.etB), (const unsigned long long*)(ws + L.colbits),
                     d.np, nB);
  return hipGetLastError();
}

hipError_t oz2_launch_scales(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                             uint8_t* ws, int side, hipStream_t s) {
  unsigned blocks = (unsigned)((d.mp + d.np + 255) / 256);
  hipLaunchKernelGGL(k_scales, dim3(blocks), dim3(256), 0, s, d,
                     (const unsigned long long*)(ws + L.rowbits),
                     (const unsigned long long*)(ws + L.colbits), (const uint32_t*)(ws + L.Rmax),
                     (const uint32_t*)(ws + L.Kmax), (int32_t*)(ws + L.sA), (int32_t*)(ws + L.tB),
                     (int32_t*)(ws + L.eA), (int32_t*)(ws + L.eB), (uint32_t*)(ws + L.flagsA), (uint32_t*)(ws + L.flagsB), c.cA, c.cB,
                     (int*)(ws + L.counters), (int*)(ws + L.listA), (int*)(ws + L.listB), side);
  return hipGetLastError();
}

hipError_t oz2_launch_tables(const Oz2Layout& L, const Oz2Const& c, uint8_t* ws, hipStream_t s) {
  hipLaunchKernelGGL(k_plane_tables, dim3((c.tabsz + 255) / 256), dim3(256), 0, s, c,
                     (uint32_t*)(ws + L.tabs));
  return hipGetLastError();
}

// workgroups of k_split that stay resident on the whole device for a given
// LDS table size (cached per size under a lock: the size depends only on r)
static int split_resident(size_t lds) {
  static std::mutex mu;
  static int cache_lds[OZ2_MAXR + 1] = {0}, cache_n[OZ2_MAXR + 1] = {0};
  std::lock_guard<std::mutex> g(mu);
  const int slot = (int)(lds % (OZ2_MAXR + 1));
  if (cache_lds[slot] == (int)lds) return cache_n[slot];
  // dynamic LDS above 64 KiB (tables for r = 16 plus the staged tile) must be opted into
  (void)hipFuncSetAttribute((const void*)k_split, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_split, 256, lds) !=
          hipSuccess ||
      per_cu <= 0)
    per_cu = 1;
  cache_lds[slot] = (int)lds;
  cache_n[slot] = per_cu * oz2_device_cus();
  return cache_n[slot];
}

hipError_t oz2_launch_split(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                            const double* A, int lda, const double* B, int ldb, int side,
                            hipStream_t s) {
  unsigned tz = (d.flags & 4u) ? 1u : 0u;   // OZ2_QUANT_TZ
  const int listed = (d.flags & 16u) ? 1 : 0;   // OZ2_FORCE_FALLBACK
  const size_t lds = (size_t)c.tabsz * 4;
  SplitSide SA{A, lda, d.m, d.mp, d.mp / 64, 0, (const int32_t*)(ws + L.sA),
               (uint32_t*)(ws + L.flagsA), ws + L.planesA, 0u, (int*)(ws + L.counters),
               (int*)(ws + L.listA), listed};
  SplitSide SB{B, ldb, d.n, d.np, d.np / 64, 0, (const int32_t*)(ws + L.tB),
               (uint32_t*)(ws + L.flagsB), ws + L.planesB,
               ((uintptr_t)B % 16 == 0 && ldb % 2 == 0) ? 1u : 0u, (int*)(ws + L.counters) + 1,
               (int*)(ws + L.listB), listed};
  if (side & OZ2_SIDE_A) SA.ntiles = (d.mp / 64) * (d.kp / 64);
  if (side & OZ2_SIDE_B) SB.ntiles = (d.np / 64) * (d.kp / 64);
  const int total = SA.ntiles + SB.ntiles, cap = split_resident(lds);
  if (total == 0) return hipSuccess;
  // persistent-style grid: one resident round of workgroups walks the tiles
  hipLaunchKernelGGL(k_split, dim3(total < cap ? total : cap), dim3(256), lds, s, c, SA, SB, d.k,
                     d.kp, (const uint32_t*)(ws + L.tabs), tz);
  return hipGetLastError();
}
