// Many small products in one launch (m, n, k <= 64): the whole of Alg. 1 --
// scan, max-magnitude codes and their FP8 product, scales, quantise, residue
// planes, the 3r FP8 residue products with exact FP32 chains, CRT
// reconstruction with one rounding, and the native-FP64 fallback -- runs
// inside one workgroup per problem, with the digit planes in LDS and the
// residues in registers.  Nothing is staged through HBM: the kernel reads A
// and B and writes C.
//
// Workgroup: 512 threads (8 waves).  Thread t owns row t/8 of A (column t/8
// of B) and k chunk 8 (t%8) .. +7 for the scan, codes and planes.  Wave w
// owns the two 16 x 16 output blocks at block row w/2, block columns
// 2 (w%2) and 2 (w%2) + 1: v_mfma_f32_16x16x128_f8f6f4 with K = 128
// (k <= 64 real, the rest zero), one per block and plane product, so each
// lane ends with 8 outputs (one uint4 of int16 residues per modulus).
// Persistent grid: each workgroup walks problems b = blockIdx.x, += gridDim.x.
#include "oz2_device.h"

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int PP = 80;   // bytes per plane row (64 + 16: spreads the LDS banks)
constexpr int NTB = 512;

struct Smem {
  // the quantised chunks of A and B: a = h 2^32 + l; elements j, j + 1 of
  // thread t's chunk as one int4 (h_j, l_j, h_j+1, l_j+1) at [j / 2][t], so
  // that a wave's 16-byte accesses are contiguous (no bank conflicts);
  // written once per problem and read for every modulus
  int4 qa[4][NTB];
  int4 qb[4][NTB];
  uint8_t pa[3][64][PP];
  uint8_t pb[4][64][PP];     // B: d0, d1, d0 + d1 and, for nonsquare moduli, -16 d1
  unsigned long long rbits[64], cbits[64];
  uint32_t Rm[64], Km[64];
  int sS[64], sT[64];
  uint32_t fA[64], fB[64];
};

// max over the 8 lanes of a row group (lanes 8g .. 8g+7)
__device__ __forceinline__ unsigned long long oct_max(unsigned long long v) {
  for (int o = 1; o <= 4; o <<= 1) {
    const unsigned long long u = (unsigned long long)__shfl_xor((long long)v, o);
    v = v > u ? v : u;
  }
  return v;
}

// operand fragment: plane rows base + lane%16, k bytes 32 (lane/16) .. +31
// (lanes 32..63 hold k >= 64: zero)
__device__ __forceinline__ v8i frag(const uint8_t (*pl)[PP], int base) {
  const int lane = threadIdx.x & 63;
  if (lane >= 32) return v8i{0, 0, 0, 0, 0, 0, 0, 0};
  const uint8_t* p = pl[base + (lane & 15)] + 32 * (lane >> 4);
  const uint4 lo = *reinterpret_cast<const uint4*>(p);
  const uint4 hi = *reinterpret_cast<const uint4*>(p + 16);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// two operands in one: k 0..63 of plane `lo` in lanes 0..31 and k 0..63 of
// plane `hi` in lanes 32..63 (the instruction's K = 128), so one MFMA sums
// the products of both pairs
__device__ __forceinline__ v8i frag2(const uint8_t (*lo)[PP], const uint8_t (*hi)[PP], int base) {
  const int lane = threadIdx.x & 63;
  const uint8_t* p = (lane < 32 ? lo : hi)[base + (lane & 15)] + 32 * ((lane >> 4) & 1);
  const uint4 l4 = *reinterpret_cast<const uint4*>(p);
  const uint4 h4 = *reinterpret_cast<const uint4*>(p + 16);
  return v8i{(int)l4.x, (int)l4.y, (int)l4.z, (int)l4.w, (int)h4.x, (int)h4.y, (int)h4.z, (int)h4.w};
}

__device__ __forceinline__ v4f mfma(v8i a, v8i b, v4f c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// Quantise (Eq. (scale)) the thread's chunk (8 consecutive k of one row,
// already zero for T1 rows) once per problem: a = rint(x 2^s) = h 2^32 + l
// with |h| <= 2^30 (|a| <= 2^62) and 0 <= l < 2^32, stored as (h, l) in LDS
// (q[j / 2][thread]).
__device__ __forceinline__ void quantise8(const double (&x)[8], int sc, bool& t2,
                                          int4 (*q)[NTB]) {
#pragma unroll
  for (int j = 0; j < 8; j += 2) {
    int2 v[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const double a = rint(ldexp(x[j + u], sc));
      t2 |= (x[j + u] != 0.0) && (a == 0.0);
      const double hd = floor(a * 0x1p-32);
      v[u] = make_int2((int)hd, (int)(uint32_t)fma(-hd, 0x1p32, a));
    }
    q[j >> 1][threadIdx.x] = make_int4(v[0].x, v[0].y, v[1].x, v[1].y);
  }
}

// 8 plane bytes of this thread's quantised chunk into the planes of modulus i
// (FOUR: also the -16 d1 plane of a nonsquare modulus, for B)
template <bool FOUR>
__device__ __forceinline__ void split8(const Oz2Const& c, int i, const uint32_t* tab,
                                       const int4 (*q)[NTB], uint8_t (*pl)[64][PP], int row,
                                       int ch) {
  const double m = (double)c.m[i], c32 = (double)c.c32[i], dinv = c.dinv[i];
  const int to = c.toff[i];
  uint32_t e[8];
#pragma unroll
  for (int j = 0; j < 8; j += 2) {
    const int4 hl = q[j >> 1][threadIdx.x];
    e[j] = tab[to + centred_residue((double)hl.x, (double)(uint32_t)hl.y, m, c32, dinv)];
    e[j + 1] = tab[to + centred_residue((double)hl.z, (double)(uint32_t)hl.w, m, c32, dinv)];
  }
  uint2 v0, v1;
  v0.x = gather_byte(e[0], e[1], e[2], e[3], 0x05010400u);
  v0.y = gather_byte(e[4], e[5], e[6], e[7], 0x05010400u);
  v1.x = gather_byte(e[0], e[1], e[2], e[3], 0x05010501u);
  v1.y = gather_byte(e[4], e[5], e[6], e[7], 0x05010501u);
  *reinterpret_cast<uint2*>(&pl[0][row][ch]) = v0;
  *reinterpret_cast<uint2*>(&pl[1][row][ch]) = v1;
  if (!c.sq[i]) {
    uint2 v2;
    v2.x = gather_byte(e[0], e[1], e[2], e[3], 0x05010602u);
    v2.y = gather_byte(e[4], e[5], e[6], e[7], 0x05010602u);
    *reinterpret_cast<uint2*>(&pl[2][row][ch]) = v2;
    if (FOUR) {
      uint2 v3;
      v3.x = gather_byte(e[0], e[1], e[2], e[3], 0x05010703u);
      v3.y = gather_byte(e[4], e[5], e[6], e[7], 0x05010703u);
      *reinterpret_cast<uint2*>(&pl[3][row][ch]) = v3;
    }
  }
}

// The three plane products of modulus i for the wave's two blocks (the
// chains of the residue GEMM): acc[q][e] is output 4q + e, an exact integer
// below 2^16 in magnitude, congruent to C~ / fin mod m.
__device__ __forceinline__ void modulus_chain(const Oz2Const& c, int i, const Smem& S, int rb0,
                                              int cb0, v4f (&acc)[2]) {
  const int m = c.m[i], s = c.sq[i];
  const float fm = (float)m, inv = c.finv[i];
  auto reduce_mul = [&](v4f v, float rho) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = __builtin_fmaf(-rintf(v[e] * inv), fm, v[e]) * rho;
    return v;
  };
  acc[0] = v4f{0.f};
  acc[1] = v4f{0.f};
  if (s) {          // (d1 e0 + d0 e1) x s + d0 e0, the cross pair in one MFMA
    const v8i a10 = frag2(S.pa[1], S.pa[0], rb0), a0 = frag(S.pa[0], rb0);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      acc[q] = mfma(a10, frag2(S.pb[0], S.pb[1], cb0 + 16 * q), acc[q]);
      acc[q] = reduce_mul(acc[q], (float)s);
      acc[q] = mfma(a0, frag(S.pb[0], cb0 + 16 * q), acc[q]);
    }
  } else {          // (d1 (-16 e1) + d0 e0) x rho1 + (d0+d1)(e0+e1), then x 16
    // (-16 = 240 / -15 mod m; the first pair in one MFMA, exact for k <= 64:
    // |sum| < 2^19)
    const v8i a10 = frag2(S.pa[1], S.pa[0], rb0), a2 = frag(S.pa[2], rb0);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      acc[q] = mfma(a10, frag2(S.pb[3], S.pb[0], cb0 + 16 * q), acc[q]);
      acc[q] = reduce_mul(acc[q], (float)c.rho1[i]);
      acc[q] = mfma(a2, frag(S.pb[2], cb0 + 16 * q), acc[q]);
    }
  }
}

// The centred residues of the 8 outputs of modulus i, two per word: word q
// holds outputs 2q, 2q+1 (output = 4 block + e).
__device__ __forceinline__ uint4 modulus_products(const Oz2Const& c, int i, const Smem& S, int rb0,
                                                  int cb0) {
  const int m = c.m[i];
  const float fm = (float)m, inv = c.finv[i];
  v4f acc[2];
  modulus_chain(c, i, S, rb0, cb0, acc);
  const int fin = c.fin[i];
  int rr[8];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v = acc[q][e];
      if (fin != 1) v = __builtin_fmaf(-rintf(v * inv), fm, v) * (float)fin;
      rr[4 * q + e] = oz2_centre((int)v, m, inv);
    }
  uint32_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) w[q] = ((uint32_t)rr[2 * q] & 0xFFFFu) | ((uint32_t)rr[2 * q + 1] << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// r <= 12: output 4q + e's residue of modulus i, reduced once, added into its
// CRT sums.  The chain value v (|v| < 2^16, exact) is congruent to C~/fin mod
// m; reduced with the fp32 quotient estimate it lies within m/2 + 1 of zero,
// and the sums take it times the weights of fin W_i (W38f), which gives the
// same integers mod M as fin v times W_i.  Any representative of magnitude
// <= 577 serves the sums, whose limbs stay below 2^52.
__device__ __forceinline__ void crt_add(const Oz2Const& c, int i, const v4f (&acc)[2],
                                        double (&S0)[8], double (&S1)[8], double (&S2)[8]) {
  const float fm = (float)c.m[i], inv = c.finv[i];
  const double w0 = c.W38f[i][0], w1 = c.W38f[i][1], w2 = c.W38f[i][2];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float v = acc[q][e];
      const double x = (double)__builtin_fmaf(-rintf(v * inv), fm, v);
      const int I = 4 * q + e;
      S0[I] = fma(x, w0, S0[I]);
      S1[I] = fma(x, w1, S1[I]);
      S2[I] = fma(x, w2, S2[I]);
    }
}

// r <= 12: the lane's eight outputs (output I at row rb0 + 4 (lane/16) + I%4,
// column cb0 + 16 (I/4) + lane%16) from their CRT sums: reduction by the
// quotient estimate, one rounding with the exponent shift; flagged rows and
// columns recomputed in native FP64; only outputs inside m x n stored.
// With iout (a diagnostic probe) the exact integers of the unflagged outputs
// are written there instead, 5 words each at [col][row] of the problem's
// m x n block, and C is not touched.
__device__ __forceinline__ void emit38(const Oz2Const& c, const double (&S0)[8],
                                       const double (&S1)[8], const double (&S2)[8],
                                       const Smem& S, int rb0, int cb0, int m, int n, int k,
                                       const double* __restrict__ A, int lda,
                                       const double* __restrict__ B, int ldb, double* C, int ldc,
                                       uint32_t* iout) {
  const int lane = threadIdx.x & 63;
  const int r0 = rb0 + 4 * (lane >> 4), c0 = cb0 + (lane & 15);
#pragma unroll
  for (int I = 0; I < 8; ++I) {
    const int row = r0 + (I & 3), col = c0 + 16 * (I >> 2);
    if (row < m && col < n) {
      const bool flagged = ((S.fA[row] | S.fB[col]) & (OZ2_T1 | OZ2_T2)) != 0;
      if (iout) {
        if (!flagged) {
          double s[3] = {S0[I], S1[I], S2[I]};
          if (crt38_reduce<3>(c, s)) crt38_fix<3>(c, s);
          uint32_t w[4];
          limbs38_words<3>(s, w);
          uint32_t* o = iout + ((size_t)col * m + row) * NL;
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = w[q];
          o[4] = (uint32_t)((int32_t)w[3] >> 31);
        }
        continue;
      }
      double v;
      if (flagged) {
        double sacc = 0.0;   // native FP64, one FMA per k in ascending k
        for (int l = 0; l < k; ++l) sacc = fma(A[row + (size_t)l * lda], B[l + (size_t)col * ldb], sacc);
        v = sacc;
      } else {
        double s[3] = {S0[I], S1[I], S2[I]};
        if (crt38_reduce<3>(c, s)) crt38_fix<3>(c, s);
        v = round38<3>(s, S.sS[row] + S.sT[col]);
      }
      C[row + (size_t)col * ldc] = v;
    }
  }
}

// res[i] = v for a runtime i without dynamic register indexing
template <int R>
__device__ __forceinline__ void put_res(uint4 (&res)[R], int i, uint4 v) {
#pragma unroll
  for (int q = 0; q < R; ++q)
    if (q == i) res[q] = v;
}

template <int R, int I>
struct Emit {
  __device__ __forceinline__ static void run(const Oz2Const& c, const uint4 (&x)[R],
                                             const Smem& S, int rb0, int cb0, int m, int n, int k,
                                             const double* __restrict__ A, int lda,
                                             const double* __restrict__ B, int ldb, double* C,
                                             int ldc, uint32_t* iout) {
    constexpr int NW = NWords<R>::value;
    const int lane = threadIdx.x & 63;
    const int row = rb0 + 4 * (lane >> 4) + (I & 3);
    const int col = cb0 + 16 * (I >> 2) + (lane & 15);
    if (row < m && col < n) {
      const bool flagged = ((S.fA[row] | S.fB[col]) & (OZ2_T1 | OZ2_T2)) != 0;
      if (iout) {
        if (!flagged) {
          uint32_t w[NW];
          crt_words<R, NW, I>(c, x, w);
          uint32_t* o = iout + ((size_t)col * m + row) * NL;
#pragma unroll
          for (int q = 0; q < NL; ++q) o[q] = q < NW ? w[q < NW ? q : 0] : (uint32_t)((int32_t)w[NW - 1] >> 31);
        }
      } else {
        double v;
        if (flagged) {
          double sacc = 0.0;   // native FP64, one FMA per k in ascending k
          for (int l = 0; l < k; ++l) sacc = fma(A[row + (size_t)l * lda], B[l + (size_t)col * ldb], sacc);
          v = sacc;
        } else {
          uint32_t w[NW];
          crt_words<R, NW, I>(c, x, w);
          v = round_scaled<NW>(w, S.sS[row] + S.sT[col]);
        }
        C[row + (size_t)col * ldc] = v;
      }
    }
    Emit<R, I + 1>::run(c, x, S, rb0, cb0, m, n, k, A, lda, B, ldb, C, ldc, iout);
  }
};
template <int R>
struct Emit<R, 8> {
  __device__ __forceinline__ static void run(const Oz2Const&, const uint4 (&)[R], const Smem&, int,
                                             int, int, int, int, const double*, int, const double*,
                                             int, double*, int, uint32_t*) {}
};

// INT (a diagnostic instantiation): write the exact integers to iout instead
// of C; the product path runs INT = false, where iout is not used at all.
template <int R, bool INT>
__global__ void __launch_bounds__(NTB)
k_batched(Oz2Const c, int m, int n, int k, int batch, const double* __restrict__ A, int lda,
          long long strideA, const double* __restrict__ B, int ldb, long long strideB, double* C,
          int ldc, long long strideC, const uint32_t* __restrict__ gtab, uint32_t* iout) {
  extern __shared__ uint32_t tab[];
  __shared__ __attribute__((aligned(16))) Smem S;
  for (int i = threadIdx.x; i < c.tabsz; i += blockDim.x) tab[i] = gtab[i];
  const int t = threadIdx.x, row = t >> 3, ch = (t & 7) * 8;
  const int w = t >> 6, lane = t & 63;
  const int rb0 = 16 * (w >> 1), cb0 = 32 * (w & 1);
  for (int b = blockIdx.x; b < batch; b += gridDim.x) {
    const double* Ab = A + (size_t)b * strideA;
    const double* Bb = B + (size_t)b * strideB;
    double* Cb = C + (size_t)b * strideC;
    uint32_t* Ib = INT ? iout + (size_t)b * m * n * NL : nullptr;
    __syncthreads();   // the previous problem (and the table copy) are done with S
    // scan: row maxima of |A|, column maxima of |B| (bit patterns), T1
    double xa[8], xb[8];
    unsigned long long ma = 0, mb = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int l = ch + j;
      xa[j] = (row < m && l < k) ? Ab[row + (size_t)l * lda] : 0.0;
      xb[j] = (row < n && l < k) ? Bb[l + (size_t)row * ldb] : 0.0;
      ma = max(ma, abs_bits(xa[j]));
      mb = max(mb, abs_bits(xb[j]));
    }
    ma = oct_max(ma);
    mb = oct_max(mb);
    if ((t & 7) == 0) {
      S.rbits[row] = ma;
      S.cbits[row] = mb;
      S.Rm[row] = 0;
      S.Km[row] = 0;
      S.fA[row] = ma >= kInfBits ? OZ2_T1 : 0u;
      S.fB[row] = mb >= kInfBits ? OZ2_T1 : 0u;
    }
    const bool t1a = ma >= kInfBits, t1b = mb >= kInfBits;
    const int Ea = (ma == 0 || t1a) ? 0 : exp_of_bits(ma);
    const int Eb = (mb == 0 || t1b) ? 0 : exp_of_bits(mb);
    // 4-bit magnitude codes into plane 0
    {
      uint2 va, vb;
      va.x = t1a ? 0u : pack4_fp8(code_of(xa[0], Ea), code_of(xa[1], Ea), code_of(xa[2], Ea),
                                  code_of(xa[3], Ea));
      va.y = t1a ? 0u : pack4_fp8(code_of(xa[4], Ea), code_of(xa[5], Ea), code_of(xa[6], Ea),
                                  code_of(xa[7], Ea));
      vb.x = t1b ? 0u : pack4_fp8(code_of(xb[0], Eb), code_of(xb[1], Eb), code_of(xb[2], Eb),
                                  code_of(xb[3], Eb));
      vb.y = t1b ? 0u : pack4_fp8(code_of(xb[4], Eb), code_of(xb[5], Eb), code_of(xb[6], Eb),
                                  code_of(xb[7], Eb));
      *reinterpret_cast<uint2*>(&S.pa[0][row][ch]) = va;
      *reinterpret_cast<uint2*>(&S.pb[0][row][ch]) = vb;
    }
    __syncthreads();
    // the max-magnitude product G' = codesA codesB^T (exact: <= 256 k) and its
    // row / column maxima; lane holds rows rb0 + 4 (lane/16) + e, column lane%16
    {
      const v8i a = frag(S.pa[0], rb0);
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const v4f g = mfma(a, frag(S.pb[0], cb0 + 16 * q), v4f{0.f});
        float cmax = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float v = g[e];
          cmax = fmaxf(cmax, v);
          for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o));
          if ((lane & 15) == 0) atomicMax(&S.Rm[rb0 + 4 * (lane >> 4) + e], (uint32_t)v);
        }
        cmax = fmaxf(cmax, __shfl_xor(cmax, 16));
        cmax = fmaxf(cmax, __shfl_xor(cmax, 32));
        if (lane < 16) atomicMax(&S.Km[cb0 + 16 * q + lane], (uint32_t)cmax);
      }
    }
    __syncthreads();
    if (t < 64) {
      const unsigned long long bb = S.rbits[t];
      int s = 0;
      if (t < m && bb < kInfBits) s = width_of(S.Rm[t], c.cA) - (bb ? exp_of_bits(bb) : 0);
      S.sS[t] = s;
    } else if (t < 128) {
      const int j = t - 64;
      const unsigned long long bb = S.cbits[j];
      int s = 0;
      if (j < n && bb < kInfBits) s = width_of(S.Km[j], c.cB) - (bb ? exp_of_bits(bb) : 0);
      S.sT[j] = s;
    }
    __syncthreads();
    // the thread's chunks, quantised once (T1 rows and columns as zeros); the
    // thread reads back only its own chunk, so no barrier is needed here
    bool t2a = false, t2b = false;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      xa[j] = t1a ? 0.0 : xa[j];
      xb[j] = t1b ? 0.0 : xb[j];
    }
    quantise8(xa, S.sS[row], t2a, S.qa);
    quantise8(xb, S.sT[row], t2b, S.qb);
    // The workgroup's next problem: one 8-byte load per thread touches each
    // of its 128-byte lines of A (threads 0..255: column t/4, rows 16 (t%4)
    // ..) and B (threads 256..511), so that they sit in L2 when that problem
    // starts (its loads are otherwise the only memory latency a problem
    // exposes).  The value is consumed by an empty asm after this problem's
    // outputs are written: no effect on the results.
    double touch = 0.0;
    {
      const size_t bn = (size_t)b + gridDim.x;
      const int tl = t & 255, col = tl >> 2, seg = 16 * (tl & 3);
      if (bn < (size_t)batch) {
        if (t < 256 && col < k && seg < m) touch = A[bn * strideA + (size_t)col * lda + seg];
        if (t >= 256 && col < n && seg < k) touch = B[bn * strideB + (size_t)col * ldb + seg];
      }
    }
    if constexpr (R <= 12) {
      // each modulus's residues go straight into the CRT sums (three
      // radix-2^38 limbs per output)
      double S0[8], S1[8], S2[8];
#pragma unroll
      for (int I = 0; I < 8; ++I) S0[I] = S1[I] = S2[I] = 0.0;
#pragma nounroll
      for (int i = 0; i < R; ++i) {
        split8<false>(c, i, tab, S.qa, S.pa, row, ch);
        split8<true>(c, i, tab, S.qb, S.pb, row, ch);
        __syncthreads();
        v4f acc[2];
        modulus_chain(c, i, S, rb0, cb0, acc);
        crt_add(c, i, acc, S0, S1, S2);
        __syncthreads();
      }
      if (t2a && row < m) atomicOr(&S.fA[row], OZ2_T2);
      if (t2b && row < n) atomicOr(&S.fB[row], OZ2_T2);
      __syncthreads();
      emit38(c, S0, S1, S2, S, rb0, cb0, m, n, k, Ab, lda, Bb, ldb, Cb, ldc, Ib);
      asm volatile("" ::"v"(touch));
    } else {
      // residues of every modulus: one uint4 (8 int16 outputs) per modulus
      uint4 res[R];
#pragma nounroll
      for (int i = 0; i < R; ++i) {
        split8<false>(c, i, tab, S.qa, S.pa, row, ch);
        split8<true>(c, i, tab, S.qb, S.pb, row, ch);
        __syncthreads();
        put_res<R>(res, i, modulus_products(c, i, S, rb0, cb0));
        __syncthreads();
      }
      if (t2a && row < m) atomicOr(&S.fA[row], OZ2_T2);
      if (t2b && row < n) atomicOr(&S.fB[row], OZ2_T2);
      __syncthreads();
      Emit<R, 0>::run(c, res, S, rb0, cb0, m, n, k, Ab, lda, Bb, ldb, Cb, ldc, Ib);
      asm volatile("" ::"v"(touch));
    }
  }
}

template <int R>
hipError_t launch_r(const Oz2Const& c, int m, int n, int k, int batch, const double* A, int lda,
                    long long sA, const double* B, int ldb, long long sB, double* C, int ldc,
                    long long sC, const uint32_t* tab, uint32_t* iout, hipStream_t s) {
  const size_t lds = (size_t)c.tabsz * 4;
  const int cus = oz2_device_cus();
  auto kern = iout ? k_batched<R, true> : k_batched<R, false>;
  (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
  int per = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kern, NTB, lds) != hipSuccess ||
      per < 1)
    per = 1;
  const int grid = min(batch, per * cus);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(NTB), lds, s, c, m, n, k, batch, A, lda, sA,
                     B, ldb, sB, C, ldc, sC, tab, iout);
  return hipGetLastError();
}

}  // namespace

hipError_t oz2_launch_batched(const Oz2Const& c, int m, int n, int k, int batch, const double* A,
                              int lda, long long sA, const double* B, int ldb, long long sB,
                              double* C, int ldc, long long sC, const uint32_t* tab,
                              uint32_t* iout, hipStream_t s) {
  switch (c.r) {
    case 8: return launch_r<8>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    case 9: return launch_r<9>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    case 10: return launch_r<10>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    case 11: return launch_r<11>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    case 12: return launch_r<12>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    case 13: return launch_r<13>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    case 14: return launch_r<14>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    case 15: return launch_r<15>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    case 16: return launch_r<16>(c, m, n, k, batch, A, lda, sA, B, ldb, sB, C, ldc, sC, tab, iout, s);
    default: return hipErrorInvalidValue;
  }
}
