// Batched GEMV Y = A X (X: k x nrhs, nrhs <= 16) as the paper's fused Ozaki-II
// GEMV (Alg. 2, section "Strategy 1: Batched GEMV"): every element of A is
// read once in FP64 and deconstructed on the fly -- quantised with its row's
// scale, reduced modulo each m_i, split into E4M3 digit planes -- and the
// planes of every modulus go straight into FP8 MFMAs against the planes of X,
// with all r sets of accumulators held in registers (the paper's
// C_acc^(1..r)).  Nothing of A is written back.  The scaling diagonals D, E
// are inputs of Alg. 2; here they are the fixed rule of Alg. 1's bound
// mu = k max|A~| max|X~| (OZ2_SCALE_FIXED: a row's scale depends on that row
// alone), computed by the staged path's scan and scale kernels.
//
// Kernels (after the scan and scale kernels and the plane tables):
//  * k_gemv_xplanes: X quantised, reduced and split once into MFMA operand
//    fragments [chunk][plane][half][lane][16 B] (k in chunks of 128);
//  * k_gemv<R>: a workgroup of 8 waves (2 per SIMD) owns 128 rows of A (wave
//    w rows 16w..16w+15) and a range of chunks (split-K); per 32-k quarter of
//    a chunk each lane loads 8 elements of its row (row L%16, k 8(L/16)..+7:
//    exactly its operand bytes of v_mfma_f32_16x16x32_fp8_fp8), the next
//    quarter's loads in flight, quantises them once, then per modulus forms
//    their residues (exact fp64), looks the E4M3 plane bytes up in an LDS
//    table and issues the modulus's three plane products against the X
//    fragments (staged in LDS, shared by the 8 waves).  Square m = s^2:
//    acc0 += d0 e0, acc1 += d1 e0 + d0 e1; nonsquare (Eq. (kar), b = 4):
//    acc0 += (d0+d1)(e0+e1), acc1 += d0 e0, acc2 += d1 e1.  Every partial
//    sum is an integer below 2^24 while a split spans at most 32768 k
//    (Eq. (accum-exact)).  The epilogue combines them with the coefficients
//    (1, s) or (16, -15, 240) modulo m and stores a representative per
//    output and modulus (int16, |x| <= m/2 + 2);
//  * k_gemv_crt<R>: sums the splits' residues modulo m, reconstructs the
//    exact integer with the reconstruction's own CRT routine, rounds it once
//    with the shift -(s_i + t_b) and writes Y (rows and columns flagged for
//    the native fallback are left to it).
#include "oz2_device.h"

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int GV_ROWS = 128;   // rows of A per workgroup
constexpr int GV_K = 128;      // k per chunk (X's fragments are staged per chunk)
constexpr int GV_NT = 512;     // threads per workgroup (8 waves)
constexpr int GV_FRAG = 2048;  // bytes of one plane's operand fragments per chunk

// 16 x 16 x 32 E4M3 product: lane L holds row (A) / column (B) L%16,
// k 8(L/16) .. +7; the result lane L column L%16, rows 4(L/16) .. +3
__device__ __forceinline__ v4f mfma16k32(long a, long b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_fp8_fp8(a, b, c, 0, 0, 0);
}

// Quantise 32 elements with the power-of-two scale sc (Eq. (scale)): a =
// RN(x 2^sc) (or truncation) = ah 2^32 + al, exact; t2 is set when a nonzero
// element quantises to zero.
__device__ __forceinline__ void quantise32(const double (&x)[32], int sc, unsigned tz, bool& t2,
                                           double (&ah)[32], double (&al)[32]) {
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    const double y = ldexp(x[j], sc);
    const double a = tz ? trunc(y) : rint(y);
    t2 |= (x[j] != 0.0) && (a == 0.0);
    const double h = floor(a * 0x1p-32);
    ah[j] = h;
    al[j] = fma(-h, 0x1p32, a);
  }
}

// Operand bytes of the planes of modulus i for 32 quantised elements: word g
// of plane p holds the E4M3 digit bytes of elements 4g..4g+3 (table entry
// byte p: d0, d1, d0 + d1).
template <bool SQ>
__device__ __forceinline__ void planes32(const Oz2Const& c, int i, const uint32_t* tab,
                                         const double (&ah)[32], const double (&al)[32],
                                         v8i& p0, v8i& p1, v8i& p2) {
  const double m = (double)c.m[i], c32 = (double)c.c32[i], dinv = c.dinv[i];
  const int to = c.toff[i];
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    uint32_t e[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) e[u] = tab[to + centred_residue(ah[4 * g + u], al[4 * g + u], m, c32, dinv)];
    p0[g] = (int)gather_byte(e[0], e[1], e[2], e[3], 0x05010400u);
    p1[g] = (int)gather_byte(e[0], e[1], e[2], e[3], 0x05010501u);
    if (!SQ) p2[g] = (int)gather_byte(e[0], e[1], e[2], e[3], 0x05010602u);
  }
}

// Quantise 8 elements (as quantise32).
__device__ __forceinline__ void quantise8(const double (&x)[8], int sc, unsigned tz, bool& t2,
                                          double (&ah)[8], double (&al)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const double y = ldexp(x[j], sc);
    const double a = tz ? trunc(y) : rint(y);
    t2 |= (x[j] != 0.0) && (a == 0.0);
    const double h = floor(a * 0x1p-32);
    ah[j] = h;
    al[j] = fma(-h, 0x1p32, a);
  }
}

// Operand bytes of the planes of modulus i for 8 quantised elements (byte j
// of plane p: table entry byte p of element j: d0, d1, d0 + d1).
template <bool SQ>
__device__ __forceinline__ void planes8(const Oz2Const& c, int i, const uint32_t* tab,
                                        const double (&ah)[8], const double (&al)[8], long& p0,
                                        long& p1, long& p2) {
  const double m = (double)c.m[i], c32 = (double)c.c32[i], dinv = c.dinv[i];
  const int to = c.toff[i];
  uint32_t e[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) e[j] = tab[to + centred_residue(ah[j], al[j], m, c32, dinv)];
  auto word = [&](int g, uint32_t sel) { return gather_byte(e[4 * g], e[4 * g + 1], e[4 * g + 2], e[4 * g + 3], sel); };
  p0 = (long)(((uint64_t)word(1, 0x05010400u) << 32) | word(0, 0x05010400u));
  p1 = (long)(((uint64_t)word(1, 0x05010501u) << 32) | word(0, 0x05010501u));
  if (!SQ) p2 = (long)(((uint64_t)word(1, 0x05010602u) << 32) | word(0, 0x05010602u));
}

// X's operand bytes of plane p for quarter q of the chunk staged in LDS:
// lane L needs column L%16, k 32 q + 8 (L/16) .. +7, which the chunk's
// fragment layout ([half][lane'][16 B], lane' holding column lane'%16, k
// 32 (lane'/16) .. +31) keeps in lane' = 16 q + L%16, byte 8 (L/16); a
// wave's 8-byte reads cover 2 x 256 contiguous bytes
__device__ __forceinline__ long xfrag8(const uint8_t* xs, int p, int q, int lane) {
  const int u = lane >> 4;
  const uint8_t* a = xs + (size_t)p * GV_FRAG + (u >> 1) * 1024 + 16 * (16 * q + (lane & 15)) + 8 * (u & 1);
  return *reinterpret_cast<const long*>(a);
}

// x - m rint(x/m) in fp32: a representative of magnitude <= m/2 + 1 for an
// integer |x| <= 2^24 (the quotient estimate is within 2^-7 of the exact one)
__device__ __forceinline__ float red32(float x, float fm, float inv) {
  return __builtin_fmaf(-rintf(x * inv), fm, x);
}

// ---------------------------------------------------------------- X planes
// Thread (chunk c, lane L) quantises column b = L%16 of X at k = 128c +
// 32(L/16) .. +31 with its scale and writes its 32 operand bytes of every
// plane.  Columns b >= nrhs and T1 columns are zeros.  T2 columns are
// flagged and listed for the native fallback (once per column).
__global__ void __launch_bounds__(256)
k_gemv_xplanes(Oz2Const c, const double* __restrict__ X, int ldx, int k, int nrhs, int chunks,
               const int32_t* __restrict__ tB, uint32_t* flagsB, int* countB, int* listB,
               int listed, const uint32_t* __restrict__ tab, unsigned tz, uint8_t* __restrict__ xf) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= chunks * 64) return;
  const int ch = t >> 6, lane = t & 63, b = lane & 15;
  const int l0 = ch * GV_K + 32 * (lane >> 4);
  const bool cok = b < nrhs;
  const uint32_t f = cok ? flagsB[b] : 0u;
  const bool zero = !cok || (f & OZ2_T1);
  double x[32];
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    const int l = l0 + j;
    x[j] = (!zero && l < k) ? X[(size_t)l + (size_t)b * ldx] : 0.0;
  }
  bool t2 = false;
  double ah[32], al[32];
  quantise32(x, zero ? 0 : tB[b], tz, t2, ah, al);
  if (t2 && !(atomicOr(flagsB + b, OZ2_T2) & (OZ2_T1 | OZ2_T2)) && !listed)
    listB[atomicAdd(countB, 1)] = b;
  uint8_t* base = xf + (size_t)ch * c.P * GV_FRAG + 16 * lane;
  for (int i = 0; i < c.r; ++i) {
    v8i p0, p1, p2;
    if (c.sq[i]) planes32<true>(c, i, tab, ah, al, p0, p1, p2);
    else planes32<false>(c, i, tab, ah, al, p0, p1, p2);
    const int np = c.sq[i] ? 2 : 3;
    for (int p = 0; p < np; ++p) {
      const v8i v = p == 0 ? p0 : (p == 1 ? p1 : p2);
      uint8_t* d = base + (size_t)(c.pbase[i] + p) * GV_FRAG;
      *reinterpret_cast<uint4*>(d) = make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]);
      *reinterpret_cast<uint4*>(d + 1024) = make_uint4((uint32_t)v[4], (uint32_t)v[5], (uint32_t)v[6], (uint32_t)v[7]);
    }
  }
}

// ---------------------------------------------------------------- fused GEMV
// grid (row blocks of 64, splits); split s covers chunks s*cps .. +cps-1.
// The moduli come in ascending order and the six squares of the set are the
// six largest, so modulus i is square exactly when i >= R - 6 (the host
// checks this against the constants before launching).
template <int R>
__global__ void __launch_bounds__(GV_NT, 1)
k_gemv(Oz2Const c, const double* __restrict__ A, int lda, int m, int k, int chunks, int cps,
       const int32_t* __restrict__ sA, uint32_t* flagsA, int* countA, int* listA, int listed,
       const uint8_t* __restrict__ xf, const uint32_t* __restrict__ gtab, unsigned tz,
       int16_t* __restrict__ part, int mp) {
  extern __shared__ __attribute__((aligned(16))) uint32_t smem[];
  uint32_t* tab = smem;
  uint8_t* xs = reinterpret_cast<uint8_t*>(smem + ((c.tabsz + 3) & ~3));
  for (int i = threadIdx.x; i < c.tabsz; i += GV_NT) tab[i] = gtab[i];
  const int split = blockIdx.y;
  const int c0 = split * cps, c1 = min(chunks, c0 + cps);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * GV_ROWS + 16 * w + (lane & 15);
  const int kq = 8 * (lane >> 4);
  const bool rok = row < m;
  const uint32_t f0 = rok ? flagsA[row] : 0u;
  const bool zero = !rok || (f0 & OZ2_T1);
  const int sc = zero ? 0 : sA[row];
  const int fbytes = c.P * GV_FRAG;
  const double* arow = A + (size_t)row;

  v4f acc[R][3];
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int q = 0; q < 3; ++q) acc[i][q] = v4f{0.f, 0.f, 0.f, 0.f};
  bool t2 = false;
  // the lane's 8 elements of quarter q of chunk ch
  auto load8 = [&](int ch, int q, double (&x)[8]) {
    const int l0 = ch * GV_K + 32 * q + kq;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int l = l0 + j;
      x[j] = (!zero && l < k) ? arow[(size_t)l * lda] : 0.0;
    }
  };
  for (int ch = c0; ch < c1; ++ch) {
    __syncthreads();   // every wave is done with the previous chunk's fragments
    const uint4* src = reinterpret_cast<const uint4*>(xf + (size_t)ch * fbytes);
    for (int q = threadIdx.x; q < fbytes / 16; q += GV_NT) reinterpret_cast<uint4*>(xs)[q] = src[q];
    __syncthreads();   // the fragments (and, at first, the tables) are in LDS
#pragma unroll 1
    for (int q = 0; q < 4; ++q) {
      double xq[8], ah[8], al[8];
      load8(ch, q, xq);
      quantise8(xq, sc, tz, t2, ah, al);
#pragma unroll
      for (int i = 0; i < R; ++i) {
        const int pb = c.pbase[i];
        long p0, p1, p2;
        if (i >= R - 6) {
          planes8<true>(c, i, tab, ah, al, p0, p1, p2);
          const long x0 = xfrag8(xs, pb, q, lane), x1 = xfrag8(xs, pb + 1, q, lane);
          acc[i][0] = mfma16k32(p0, x0, acc[i][0]);
          acc[i][1] = mfma16k32(p1, x0, acc[i][1]);
          acc[i][1] = mfma16k32(p0, x1, acc[i][1]);
        } else {
          planes8<false>(c, i, tab, ah, al, p0, p1, p2);
          const long x0 = xfrag8(xs, pb, q, lane), x1 = xfrag8(xs, pb + 1, q, lane),
                     x2 = xfrag8(xs, pb + 2, q, lane);
          acc[i][0] = mfma16k32(p2, x2, acc[i][0]);
          acc[i][1] = mfma16k32(p0, x0, acc[i][1]);
          acc[i][2] = mfma16k32(p1, x1, acc[i][2]);
        }
      }
    }
  }
  if (t2 && !(atomicOr(flagsA + row, OZ2_T2) & (OZ2_T1 | OZ2_T2)) && !listed)
    listA[atomicAdd(countA, 1)] = row;
  // epilogue: lane L holds column L%16, rows 4(L/16) + e of the wave's 16;
  // stored as [split][modulus][row block of 16][lane][4]
  const size_t tile = (size_t)blockIdx.x * (GV_ROWS / 16) + w;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const float fm = (float)c.m[i], inv = c.finv[i];
    int16_t r4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v;
      if (i >= R - 6) {
        const float s = (float)c.sq[i];
        v = red32(acc[i][0][e], fm, inv) + s * red32(acc[i][1][e], fm, inv);
      } else {
        v = 16.0f * red32(acc[i][0][e], fm, inv) - 15.0f * red32(acc[i][1][e], fm, inv) +
            240.0f * red32(acc[i][2][e], fm, inv);
      }
      r4[e] = (int16_t)(int)red32(v, fm, inv);
    }
    int16_t* dst = part + (((size_t)split * R + i) * (mp / 16) + tile) * 256 + (size_t)lane * 4;
    *reinterpret_cast<uint2*>(dst) =
        make_uint2(((uint32_t)(uint16_t)r4[0]) | ((uint32_t)(uint16_t)r4[1] << 16),
                   ((uint32_t)(uint16_t)r4[2]) | ((uint32_t)(uint16_t)r4[3] << 16));
  }
}

// ---------------------------------------------------------------- reconstruction
template <int R, int I>
struct GvOut {
  __device__ __forceinline__ static void run(const Oz2Const& c, const uint4 (&x)[R], int row0, int b,
                                             int m, int nrhs, const int32_t* __restrict__ sA,
                                             const int32_t* __restrict__ tB,
                                             const uint32_t* __restrict__ fA,
                                             const uint32_t* __restrict__ fB, bool nofb,
                                             double* Y, int ldy) {
    const int row = row0 + I;
    if (row < m && b < nrhs && (nofb || !((fA[row] | fB[b]) & (OZ2_T1 | OZ2_T2)))) {
      const int e = sA[row] + tB[b];
      double v;
      v = crt38_rounded<R, I>(c, x, e);
      Y[(size_t)row + (size_t)b * ldy] = v;
    }
    GvOut<R, I + 1>::run(c, x, row0, b, m, nrhs, sA, tB, fA, fB, nofb, Y, ldy);
  }
};
template <int R>
struct GvOut<R, 4> {
  __device__ __forceinline__ static void run(const Oz2Const&, const uint4 (&)[R], int, int, int, int,
                                             const int32_t*, const int32_t*, const uint32_t*,
                                             const uint32_t*, bool, double*, int) {}
};

// thread (row block of 16, lane): the 4 outputs of rows 4(L/16) + e, column
// L%16; the splits' representatives are summed and centred exactly
template <int R>
__global__ void __launch_bounds__(256)
k_gemv_crt(Oz2Const c, const int16_t* __restrict__ part, int splits, int mp, int m, int nrhs,
           const int32_t* __restrict__ sA, const int32_t* __restrict__ tB,
           const uint32_t* __restrict__ fA, const uint32_t* __restrict__ fB, int nofb, double* Y,
           int ldy) {
  const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t tiles = (size_t)mp / 16;
  if (t >= tiles * 64) return;
  const size_t tile = t >> 6;
  const int lane = (int)(t & 63);
  uint4 x[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    int s4[4] = {0, 0, 0, 0};
    for (int sp = 0; sp < splits; ++sp) {
      const uint2 v = *reinterpret_cast<const uint2*>(
          part + (((size_t)sp * R + i) * tiles + tile) * 256 + (size_t)lane * 4);
      s4[0] += (int16_t)(v.x & 0xFFFFu);
      s4[1] += (int16_t)(v.x >> 16);
      s4[2] += (int16_t)(v.y & 0xFFFFu);
      s4[3] += (int16_t)(v.y >> 16);
    }
    const int mi = c.m[i];
    uint32_t h[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int r = s4[e] % mi;
      r += r < 0 ? mi : 0;
      r -= r >= ((mi + 1) >> 1) ? mi : 0;   // centred: [-floor(m/2), ceil(m/2) - 1]
      h[e] = (uint32_t)(uint16_t)(int16_t)r;
    }
    x[i] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), 0u, 0u);
  }
  GvOut<R, 0>::run(c, x, (int)tile * 16 + 4 * (lane >> 4), lane & 15, m, nrhs, sA, tB, fA, fB,
                   nofb != 0, Y, ldy);
}

template <int R>
hipError_t launch_gemv_r(const Oz2Const& c, const double* A, int lda, int m, int k, int chunks,
                         int cps, int splits, const int32_t* sA, uint32_t* flagsA, int* countA,
                         int* listA, int listed, const uint8_t* xf, const uint32_t* tab,
                         unsigned tz, int16_t* part, int mp, hipStream_t s) {
  const size_t lds = (size_t)((c.tabsz + 3) & ~3) * 4 + (size_t)c.P * GV_FRAG;
  (void)hipFuncSetAttribute((const void*)k_gemv<R>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
  hipLaunchKernelGGL(k_gemv<R>, dim3(mp / GV_ROWS, splits), dim3(GV_NT), lds, s, c, A, lda, m, k,
                     chunks, cps, sA, flagsA, countA, listA, listed, xf, tab, tz, part, mp);
  return hipGetLastError();
}

template <int R>
hipError_t launch_gemv_crt_r(const Oz2Const& c, const int16_t* part, int splits, int mp, int m,
                             int nrhs, const int32_t* sA, const int32_t* tB, const uint32_t* fA,
                             const uint32_t* fB, int nofb, double* Y, int ldy, hipStream_t s) {
  const size_t threads = (size_t)mp / 16 * 64;
  hipLaunchKernelGGL(k_gemv_crt<R>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, c,
                     part, splits, mp, m, nrhs, sA, tB, fA, fB, nofb, Y, ldy);
  return hipGetLastError();
}

}  // namespace

hipError_t oz2_launch_gemv_xplanes(const Oz2Const& c, const double* X, int ldx, int k, int nrhs,
                                   const int32_t* tB, uint32_t* flagsB, int* countB, int* listB,
                                   int listed, const uint32_t* tab, unsigned tz, uint8_t* xf,
                                   hipStream_t s) {
  const int chunks = (k + GV_K - 1) / GV_K;
  const int threads = chunks * 64;
  hipLaunchKernelGGL(k_gemv_xplanes, dim3((threads + 255) / 256), dim3(256), 0, s, c, X, ldx, k,
                     nrhs, chunks, tB, flagsB, countB, listB, listed, tab, tz, xf);
  return hipGetLastError();
}

#define OZ2_GV_SWITCH(FN, ...)                      \
  switch (c.r) {                                    \
    case 8: return FN<8>(__VA_ARGS__);              \
    case 9: return FN<9>(__VA_ARGS__);              \
    case 10: return FN<10>(__VA_ARGS__);            \
    case 11: return FN<11>(__VA_ARGS__);            \
    case 12: return FN<12>(__VA_ARGS__);            \
    case 13: return FN<13>(__VA_ARGS__);            \
    case 14: return FN<14>(__VA_ARGS__);            \
    case 15: return FN<15>(__VA_ARGS__);            \
    case 16: return FN<16>(__VA_ARGS__);            \
    default: return hipErrorInvalidValue;           \
  }

hipError_t oz2_launch_gemv(const Oz2Const& c, const double* A, int lda, int m, int k, int splits,
                           const int32_t* sA, uint32_t* flagsA, int* countA, int* listA,
                           int listed, const uint8_t* xf, const uint32_t* tab, unsigned tz,
                           int16_t* part, int mp, hipStream_t s) {
  const int chunks = (k + GV_K - 1) / GV_K;
  const int cps = (chunks + splits - 1) / splits;
  OZ2_GV_SWITCH(launch_gemv_r, c, A, lda, m, k, chunks, cps, splits, sA, flagsA, countA, listA,
                listed, xf, tab, tz, part, mp, s)
}

hipError_t oz2_launch_gemv_crt(const Oz2Const& c, const int16_t* part, int splits, int mp, int m,
                               int nrhs, const int32_t* sA, const int32_t* tB, const uint32_t* fA,
                               const uint32_t* fB, int nofb, double* Y, int ldy, hipStream_t s) {
  OZ2_GV_SWITCH(launch_gemv_crt_r, c, part, splits, mp, m, nrhs, sA, tB, fA, fB, nofb, Y, ldy, s)
}
