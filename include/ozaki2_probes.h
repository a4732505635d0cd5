/* gfx950 probes behind the emulated DGEMM: the hardware facts its exactness
 * argument rests on, and the measured peaks its roofline fractions are also
 * quoted against.  Diagnostics only; the GEMM path never calls them.
 *
 * Conventions as in ozaki2.h: device pointers owned by the caller, work
 * enqueued on `stream` (a hipStream_t, NULL = default stream), status codes
 * OZ2_OK / OZ2_E_INVALID / OZ2_E_DEVICE / OZ2_E_UNSUPPORTED.
 */
#ifndef OZAKI2_PROBES_H
#define OZAKI2_PROBES_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* E4M3 (OCP E4M3FN) encoding by the conversion instruction the plane split
 * uses (v_cvt_pk_fp8_f32): out[i] = fp8(x[i]) for i < n.  x: float[n],
 * out: uint8[n], device.  The digit planes of Eq. (sq-shortcut) / Eq. (kar)
 * are exact only if every integer they hold encodes exactly; the test
 * compares this against the format's definition.  n < 0 -> OZ2_E_INVALID. */
int ozaki2_probe_e4m3(const float* x, unsigned char* out, int n, void* stream);

/* Exactness of FP32 accumulation in the FP8 MFMA (Eq. (accum-exact)): one
 * 32x32x64 E4M3 product, accumulated `chain` times into the same FP32
 * accumulator (v_mfma_f32_32x32x64_f8f6f4).  a, b: 64 lanes x 32 bytes of
 * E4M3 operand (lane L holds row / column L%32, k bytes 32(L/32)..+31),
 * out: float[64][16] accumulator registers (lane L, register e holds row
 * 8(e/4) + 4(L/32) + e%4, column L%32).  1 <= chain <= 2^20. */
int ozaki2_probe_accum(const unsigned char* a, const unsigned char* b, int chain, float* out,
                       void* stream);

/* Plain copy kernel (16 bytes per lane, grid-stride), bytes % 16 == 0 and
 * 16-byte aligned pointers; the HBM copy reference for bandwidth fractions and
 * for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE. */
int ozaki2_probe_copy(const void* src, void* dst, size_t bytes, void* stream);

/* Measured dense FP8 MFMA rate: independent 32x32x64 MFMAs on every SIMD
 * (2 waves per SIMD), timed with HIP events on an internal stream;
 * synchronous.  iters >= 1.  *tflops = FP8 TFLOP/s. */
int ozaki2_probe_mfma_peak(int iters, double* tflops);

/* Sustained FP8 MFMA rate of the residue GEMM's inner loop on plane-like
 * data: each workgroup (one per CU, 8 waves) holds 64 KiB of E4M3 bytes of
 * digits uniform in [-11, 11] in LDS; per step every wave reads its next 4 + 2
 * operand fragments from LDS while 8 MFMAs consume the current ones.  With
 * operand values toggling like the real planes the chip settles at a lower
 * clock than with the near-constant operands of ozaki2_probe_mfma_peak; the
 * residue GEMM's fractions are also quoted against this rate.  Synchronous;
 * iters >= 2 and even.  *tflops = FP8 TFLOP/s. */
int ozaki2_probe_mfma_digits(int iters, double* tflops);

/* Measured HBM copy bandwidth: copies `bytes` (>= 16 MiB) between two
 * internally allocated buffers `reps` times; synchronous; frees the buffers.
 * *gbs = (read + write bytes) / s / 1e9. */
int ozaki2_probe_copy_peak(size_t bytes, int reps, double* gbs);

/* The reconstruction's own integer and rounding routines (the direct CRT
 * sum of Eq. (garner)'s unique integer in radix-2^38 limbs, three for
 * r <= 12 and four above; one RN-even rounding) applied to n given residue
 * vectors, for tests that reach the rare branches -- integers next to +-M/2,
 * where the quotient estimate needs the exact range check -- which random
 * products almost never produce.  The residues go through the stored form
 * the reconstruction reads (x + floor(m_i/2) + 32 in a 12-bit slot) exactly
 * as the residue GEMMs write it.  residues: int16 [num_moduli][n] (modulus i
 * in ascending order; any representative x with -(floor(m_i/2) + 32) <= x <=
 * m_i/2 + 32, the range the residue GEMMs guarantee; other values give
 * undefined results but no out-of-bounds access), shifts: int [n]; words:
 * uint32 [n][5] (the integer
 * in [-M/2, M/2), two's complement, little endian), rounded: double [n]
 * (the integer times 2^-shift, rounded once).  Device pointers; asynchronous.
 * OZ2_E_INVALID for n < 0, num_moduli outside [8, 16] or a null pointer. */
int ozaki2_probe_crt(int num_moduli, const short* residues, const int* shifts, int n,
                     unsigned* words, double* rounded, void* stream);

/* The single-launch batched kernel of ozaki2_dgemm_strided_batched
 * (m, n, k <= 64) with its last step switched to writing, instead of C, the
 * exact integer it reconstructs for every output whose row and column are
 * not flagged: words = uint32 [batch][n][m][5] (device, two's complement,
 * little endian; entries of flagged rows / columns are left untouched).
 * Same A, B conventions as ozaki2_dgemm_strided_batched.  Uses the library's
 * internal workspace for the plane tables.  OZ2_E_INVALID for sizes outside
 * 1..64, a negative batch or stride, lda < m, ldb < k or a null pointer. */
int ozaki2_probe_batched_integers(int m, int n, int k, const double* A, int lda,
                                  long long strideA, const double* B, int ldb, long long strideB,
                                  int batch, int num_moduli, unsigned* words, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OZAKI2_PROBES_H */
