// Internal definitions shared by the host orchestration and the gfx950
// kernels of the Ozaki-II FP8 emulated DGEMM.  Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define OZ2_MAXR 16
#define OZ2_NLIMB 5          // 32-bit words of the exact integer: 160 bits > log2(M_max) + 1
#define OZ2_TILE 256         // output tile of the FP8 GEMMs (rows and columns)
#define OZ2_KBLK 64          // k bytes per block of the K-blocked planes = K of one
                             // v_mfma_f32_32x32x64_f8f6f4 = one GEMM stage
#define OZ2_KPAD 64          // k is padded to a multiple of this
#define OZ2_KSLAB 32768      // residue GEMM: k per exact FP32 slab, Eq. (accum-exact)
#define OZ2_FBCAP 1024       // flagged rows of A gathered into the fallback panel (at most)
#define OZ2_CSLAB 65536      // code GEMM: codes <= 16, products <= 256: 65536*256 = 2^24

// Flags per row of A / column of B.
#define OZ2_T1 1u            // a NaN or +-Inf entry
#define OZ2_T2 2u            // a nonzero entry that quantises to zero

// Per-plan constants, passed to every kernel by value (kernarg segment).
struct Oz2Const {
  int r;
  int P;                      // p_store: planes per scalar
  int m[OZ2_MAXR];            // moduli, ascending
  int sq[OZ2_MAXR];           // s if m = s^2, else 0
  int pbase[OZ2_MAXR];        // first plane of modulus i
  int c32[OZ2_MAXR];          // 2^32 mod m
  int rho0[OZ2_MAXR];         // chain transition multipliers (mod m, in [0, m))
  int rho1[OZ2_MAXR];
  int fin[OZ2_MAXR];          // final epilogue coefficient (1 square, 16 nonsquare)
  float finv[OZ2_MAXR];       // RN(1/m) in fp32
  float finv_s[OZ2_MAXR];     // RN(1/s) in fp32 (square moduli)
  double dinv[OZ2_MAXR];      // RN(1/m) in fp64
  // direct CRT sum: X = sum_i x_i W_i - q M, W_i = (M/m_i) * ((M/m_i)^-1 mod m_i)
  double W[OZ2_MAXR][OZ2_NLIMB];  // 32-bit words of W_i (exact integers in fp64)
  double wfrac[OZ2_MAXR];         // W_i / M = inv_i / m_i rounded to fp64
  double Ml[OZ2_NLIMB];           // 32-bit words of M
  double Mhalf[OZ2_NLIMB];        // 32-bit words of floor(M/2)
  int nw;                         // words of the two's complement integer in [-M/2, M/2)
  double mtop;                    // 2^(32 (nw - 1)) / M, rounded
  // the same in radix-2^38 limbs: three for r <= 12 (114 bits), four above
  // (152 bits); the reconstruction's exact integer
  double W38[OZ2_MAXR][4];
  // the same for fin_i W_i mod M = (M/m_i) ((fin_i (M/m_i)^-1) mod m_i): a
  // representative of C~/fin_i mod m_i times these gives the same sum mod M
  double W38f[OZ2_MAXR][4];
  double M38[4], Mhalf38[4];
  double mtop38;                  // 2^(38 (limbs - 1)) / M, rounded
  // the staged residues are stored as u_i = x_i + floor(m_i/2) + 32 >= 0:
  // sum_i u_i W_i limb by limb minus these gives sum_i x_i W_i exactly
  double K38[4];                  // sum_i (floor(m_i/2) + 32) W38[i][l] (exact: < 2^52)
  double Kw[OZ2_NLIMB];           // sum_i (floor(m_i/2) + 32) W[i][j] (exact: < 2^46)
  int cA, cB;                     // width budgets of the scaling rule
  // residue -> plane-bytes tables: entry toff[i] + d for the centred residue d
  int toff[OZ2_MAXR];             // (sum of the earlier moduli) + floor(m_i/2)
  int tabsz;                      // sum of the moduli (entries)
  // largest k per exact FP32 chain for which the first chain transition of
  // modulus i may be a plain multiply (x s for square m, x -16 = 240/-15 for
  // nonsquare m) without a reduction: every partial sum stays below 2^24
  int kcheap[OZ2_MAXR];
};

struct Oz2Dims {
  int m, n, k;
  int mp, np, kp;             // padded: mp, np multiples of OZ2_TILE; kp of OZ2_KPAD
  int cslabs;                 // number of code-GEMM slabs
  unsigned flags;
};

// Short k (one slab of at most 8 K-stages) on a tile count divisible by 8:
// the residue GEMMs run as two workgroups per CU and store each 32x32
// block's records pair-major (word w of lane L at 128 (w / 2) + 2 L + w % 2;
// otherwise lane-major, at 6 L + w).  Pair-major stores and loads took the
// rank-256 update's residue GEMMs and reconstruction from 11.2 / 7.8 to
// 10.9 / 7.5 ms; the long-k kernel keeps its lane-major stores.
__host__ __device__ inline bool oz2_pair_records(const Oz2Dims& d) {
  return ((d.mp / OZ2_TILE) * (d.np / OZ2_TILE)) % 8 == 0 && d.kp <= 8 * OZ2_KBLK;
}

// Workspace carve-up (byte offsets from the workspace base).
struct Oz2Layout {
  size_t rowbits, colbits;    // uint64 [mp] / [np]: max |x| bit patterns
  size_t flagsA, flagsB;      // uint32 [mp] / [np]
  size_t Rmax, Kmax;          // uint32 [cslabs][mp] / [cslabs][np]
  size_t sA, tB;              // int32 [mp] / [np]
  size_t eA, eB;              // int32 [mp] / [np]: frexp exponents of the row / column maxima
  size_t codesA, codesB;      // uint8 [kp/64][mp][64] / [kp/64][np][64] (K-blocked)
  size_t etA, etB;            // int16 [kp/64][mp] / [kp/64][np]: exponents of the tile-row maxima
  size_t planesA, planesB;    // uint8 [P][kp/64][mp][64] / [P][kp/64][np][64] (K-blocked)
  size_t tabs;                // uint32 [tabsz]: E4M3 plane bytes of every centred residue
  size_t res;                 // uint32 [r][tile][wave 8][x 4][y 2][lane 64][2][3]: per modulus
                              //   a representative x of C~ mod m_i with |x| <= m_i/2 + 32,
                              //   stored as x + floor(m_i/2) + 32 in a 12-bit slot; the 16
                              //   outputs of a lane as two 96-bit records of 8 slots
                              //   (the GEMM's accumulator order, see gemm.hip)
  size_t counters;            // int32 [4]: fallback row / column counts
  size_t listA, listB;        // int32 [mp] / [np]: flagged row / column indices
  size_t panel;               // double [k][min(mp, OZ2_FBCAP)]: the first flagged rows of A,
                              //   gathered for the native fallback (absent with NO_FALLBACK)
  size_t xfrag;               // batched GEMV: uint8 [chunks][P][2][64][16] operand fragments of X
  size_t part;                // batched GEMV: int16 [splits][r][mp/16][64][4] partial residues
  size_t total;
};

// compute units of the current device (queried once per process, thread-safe;
// 256 if the query fails)
int oz2_device_cus();

// ---------------------------------------------------------------- launchers
// Each returns hipGetLastError() of its launches.  `side` of the per-operand
// deconstruct launchers: OZ2_SIDE_A, OZ2_SIDE_B or both.
#define OZ2_SIDE_A 1
#define OZ2_SIDE_B 2
hipError_t oz2_launch_init(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, int side,
                           hipStream_t s);
hipError_t oz2_launch_scan(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws,
                           const double* A, int lda, const double* B, int ldb, int side,
                           hipStream_t s);
// scan + per-tile code bytes in one read of each operand, then the bytes
// rebased to the row exponents (the codes of the max-magnitude pass)
hipError_t oz2_launch_scan_codes(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws,
                                 const double* A, int lda, const double* B, int ldb, int side,
                                 hipStream_t s);
hipError_t oz2_launch_rebase(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, int side,
                             hipStream_t s);
hipError_t oz2_launch_codegemm(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, hipStream_t s);
hipError_t oz2_launch_scales(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                             uint8_t* ws, int side, hipStream_t s);
hipError_t oz2_launch_tables(const Oz2Layout& L, const Oz2Const& c, uint8_t* ws, hipStream_t s);
hipError_t oz2_launch_split(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                            const double* A, int lda, const double* B, int ldb, int side,
                            hipStream_t s);
hipError_t oz2_launch_resgemm(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                              uint8_t* ws, hipStream_t s);
hipError_t oz2_launch_reconstruct(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                                  uint8_t* ws, const double* A, int lda, double* C, int ldc,
                                  hipStream_t s);
hipError_t oz2_launch_fallback(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws,
                               const double* A, int lda, const double* B, int ldb,
                               double* C, int ldc, hipStream_t s);
hipError_t oz2_launch_integers(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                               uint8_t* ws, uint32_t* out, hipStream_t s);
// the reconstruction's integer and rounding routines on n given residue
// vectors (res: int16 [r][n], e: int [n] shifts; words: uint32 [n][5],
// rounded: double [n])
hipError_t oz2_launch_crt_probe(const Oz2Const& c, const int16_t* res, const int* e, int n,
                                uint32_t* words, double* rounded, hipStream_t s);
hipError_t oz2_launch_fill(double* C, int m, int n, int ldc, hipStream_t s);
// residue GEMMs and reconstruction in one kernel (fused.hip): r <= 12 and
// kp <= OZ2_KSLAB; mp, np multiples of 128 (they are of 256); C written
// (C += with OZ2_ACCUMULATE) except flagged rows / columns
hipError_t oz2_launch_fused(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                            double* C, int ldc, hipStream_t s);
// the native fallback reading A directly (no gathered panel)
hipError_t oz2_launch_fallback_direct(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws,
                                      const double* A, int lda, const double* B, int ldb,
                                      double* C, int ldc, hipStream_t s);
// batched GEMV (gemv.hip): X's operand fragments; the fused GEMV over
// `splits` k-ranges into partial residues; their reconstruction into Y
hipError_t oz2_launch_gemv_xplanes(const Oz2Const& c, const double* X, int ldx, int k, int nrhs,
                                   const int32_t* tB, uint32_t* flagsB, int* countB, int* listB,
                                   int listed, const uint32_t* tab, unsigned tz, uint8_t* xf,
                                   hipStream_t s);
hipError_t oz2_launch_gemv(const Oz2Const& c, const double* A, int lda, int m, int k, int splits,
                           const int32_t* sA, uint32_t* flagsA, int* countA, int* listA,
                           int listed, const uint8_t* xf, const uint32_t* tab, unsigned tz,
                           int16_t* part, int mp, hipStream_t s);
hipError_t oz2_launch_gemv_crt(const Oz2Const& c, const int16_t* part, int splits, int mp, int m,
                               int nrhs, const int32_t* sA, const int32_t* tB, const uint32_t* fA,
                               const uint32_t* fB, int nofb, double* Y, int ldy, hipStream_t s);
// all of Alg. 1 for `batch` problems of m, n, k <= 64 in one launch; tab = the
// residue -> plane-byte tables (oz2_launch_tables); iout (normally null, a
// diagnostic): write the exact integers of the unflagged outputs there,
// uint32 [batch][n][m][5], instead of C
hipError_t oz2_launch_batched(const Oz2Const& c, int m, int n, int k, int batch, const double* A,
                              int lda, long long sA, const double* B, int ldb, long long sB,
                              double* C, int ldc, long long sC, const uint32_t* tab, uint32_t* iout,
                              hipStream_t s);

// ---------------------------------------------------------------- digit rule
// Digit planes of a centred residue d of m (the E4M3-exact layouts of the
// "frozen plane kernel" section):
//  * square m = s^2, Eq. (sq-shortcut): balanced base-s digits
//    d0 = ((d + floor(s/2)) mod s) - floor(s/2), d1 = (d - d0)/s;
//  * nonsquare, Eq. (kar) with b = 4: balanced base-16 digits with the carry
//    correction of the "e4m3 layout envelope" paragraph (if d0+d1 is not
//    E4M3-exact -- odd and above 16 in magnitude -- move one unit of base
//    weight: (d0 - 16 sgn(d0), d1 + sgn(d0))), plus the sum plane d0+d1.
__host__ __device__ inline void oz2_digits(int d, int m, int s, int& d0, int& d1) {
  if (s) {
    const int h = s >> 1;
    int u = (d + h) % s;
    u += (u < 0) ? s : 0;
    d0 = u - h;
    d1 = (d - d0) / s;
  } else {
    d0 = ((d + 8) & 15) - 8;
    d1 = (d - d0) >> 4;
    const int sm = d0 + d1, am = sm < 0 ? -sm : sm;
    if (am > 16 && (am & 1)) {
      const int sg = d0 > 0 ? 1 : -1;
      d0 -= 16 * sg;
      d1 += sg;
    }
  }
}

// ---------------------------------------------------------------- device helpers
#ifdef __HIPCC__
// x mod m in [0, m) for |x| < 2^25 (float reciprocal estimate, one correction
// each way: the estimate of x/m is within 0.02 of the true quotient).
__device__ __forceinline__ int oz2_mod(int x, int m, float inv) {
  int q = (int)floorf((float)x * inv);
  int r = x - q * m;
  r += (r < 0) ? m : 0;
  r -= (r >= m) ? m : 0;
  return r;
}
// x - m * rint(x/m): a representative of x mod m with |result| <= m/2 + 2,
// for |x| < 2^25.
__device__ __forceinline__ int oz2_red(int x, int m, float inv) {
  int q = (int)rintf((float)x * inv);
  return x - q * m;
}
// exact centred residue in [-floor(m/2), ceil(m/2) - 1] for |x| < 2^25
__device__ __forceinline__ int oz2_centre(int x, int m, float inv) {
  int r = oz2_mod(x, m, inv);
  return (r >= ((m + 1) >> 1)) ? r - m : r;
}
#endif
