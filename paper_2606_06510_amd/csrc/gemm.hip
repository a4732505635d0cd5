// FP8 MFMA GEMMs of Alg. 1 on gfx950 (v_mfma_f32_16x16x128_f8f6f4, E4M3 x E4M3,
// FP32 accumulation):
//
//  * the max-magnitude pass ("+1" of alpha = 3r+1): G' = codesA * codesB^T,
//    epilogue = row / column maxima (integer atomics); G' is never stored;
//  * Phase 2, Eq. (modgemm): per modulus, the three E4M3 plane products of
//    Eq. (sq-shortcut) (square m = s^2: d1e0 + d0e1 with coefficient s, then
//    d0e0 with coefficient 1) or Eq. (kar) with b = 4 (nonsquare: d1e1 with
//    240, d0e0 with -15, (d0+d1)(e0+e1) with 16), accumulated exactly in FP32
//    (Eq. (accum-exact): every partial sum is an integer of magnitude
//    <= 2^24 for k <= 32768), then reduced to the centred residue.
//
// Design: one workgroup of 256 threads (4 waves) owns a 256x256 output tile;
// each wave owns 128x128 = 8x8 MFMA tiles (256 FP32 accumulators per lane).
// Operand tiles (256 rows x 128 k bytes per operand) are double buffered in
// LDS, filled by asynchronous global_load_lds (no staging registers) with an
// XOR swizzle of the 16-byte chunks so that fragment reads are bank-conflict
// free.  Per K-step: read this stage's fragments, issue the copy of the next
// stage into the other buffer, run the 64 MFMAs while it lands, then wait and
// barrier.  The three products of a modulus are run as three
// (square: two) sequential "chains" over K on ONE accumulator set: at the end
// of a chain the exact integer accumulator is reduced mod m and re-seeded as
// acc * (c_this / c_next) mod m, so the next chain continues the same
// residue.  This trades a short VALU epilogue per chain for a 256x256 tile
// (half the operand traffic of a 128x128 tile with three live accumulators).
#include "oz2_internal.h"

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int TILE = OZ2_TILE;          // 256
constexpr int KS = OZ2_KSTEP;           // 128
constexpr int OPB = TILE * KS;          // bytes of one operand stage: 32 KiB
constexpr int STAGEB = 2 * OPB;         // A + B
constexpr int LDS_BYTES = 2 * STAGEB;   // double buffered: 128 KiB

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// Asynchronous global -> LDS copy of one stage (A and B operand tiles of 256
// rows x 128 k bytes) with global_load_lds_dwordx4: each instruction writes a
// contiguous 1 KiB LDS block (lane L at +16 L), i.e. 8 tile rows; the XOR
// swizzle (physical chunk = logical chunk ^ (row & 7)) is realised by
// permuting the global addresses.  No VGPRs hold the data in flight.
__device__ __forceinline__ void issue_stage(const uint8_t* __restrict__ a,
                                            const uint8_t* __restrict__ b, int kp, int k0,
                                            uint8_t* st) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r8 = lane >> 3;
  const uint32_t lo = (uint32_t)(r8 * kp + 16 * ((lane & 7) ^ r8));   // per-lane, < 8 kp
  const uint8_t* ab = a + k0 + (size_t)(8 * w) * kp;                   // wave-uniform bases
  const uint8_t* bb = b + k0 + (size_t)(8 * w) * kp;
  lds_u8* sl = (lds_u8*)st + w * 1024;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const size_t rowj = (size_t)(32 * j) * kp;
    __builtin_amdgcn_global_load_lds((const void*)(ab + rowj + lo),
                                     (void __attribute__((address_space(3)))*)(sl + j * 4096), 16, 0, 0);
    __builtin_amdgcn_global_load_lds((const void*)(bb + rowj + lo),
                                     (void __attribute__((address_space(3)))*)(sl + OPB + j * 4096), 16, 0,
                                     0);
  }
}

__device__ __forceinline__ v8i frag(const uint8_t* p, int o0, int o1) {
  const uint4 lo = *reinterpret_cast<const uint4*>(p + o0);
  const uint4 hi = *reinterpret_cast<const uint4*>(p + o1);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// Fragments of one K-step for the wave's 128x128 sub-tile: 8 A and 8 B
// 16x128 fragments (lane -> row lane&15, k bytes 32*(lane>>4)..+31).
__device__ __forceinline__ void read_frags(const uint8_t* st, v8i (&fa)[8], v8i (&fb)[8]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wr = w >> 1, wc = w & 1;
  const int g = lane >> 4, sw = lane & 7;
  const int o0 = 16 * ((2 * g) ^ sw), o1 = 16 * ((2 * g + 1) ^ sw);
  const uint8_t* sa = st + (wr * 128 + (lane & 15)) * KS;
  const uint8_t* sb = st + OPB + (wc * 128 + (lane & 15)) * KS;
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    fa[x] = frag(sa + x * 16 * KS, o0, o1);
    fb[x] = frag(sb + x * 16 * KS, o0, o1);
  }
}

__device__ __forceinline__ void mma_stage(const v8i (&fa)[8], const v8i (&fb)[8], v4f (&acc)[8][8]) {
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b)
      acc[a][b] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(fa[a], fb[b], acc[a][b], 0, 0, 0,
                                                                  0, 0, 0);
}

// ------------------------------------------------------------- code GEMM
// grid: (tiles, code slabs).  G'[i][j] <= 256 * 65536 = 2^24: exact in FP32.
__global__ void __launch_bounds__(256, 1)
k_codegemm(const uint8_t* __restrict__ cA, const uint8_t* __restrict__ cB, int mp, int np, int kp,
           int k, uint32_t* Rmax, uint32_t* Kmax) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int ntm = mp / TILE;
  const int tile = blockIdx.x, slab = blockIdx.y;
  const int tm = tile % ntm, tn = tile / ntm;
  const int kbeg = slab * OZ2_CSLAB;
  const int kend = min(kp, kbeg + OZ2_CSLAB);
  const int nk = (kend - kbeg) / KS;
  const uint8_t* a = cA + (size_t)tm * TILE * kp;
  const uint8_t* b = cB + (size_t)tn * TILE * kp;

  v4f acc[8][8];
#pragma unroll
  for (int x = 0; x < 8; ++x)
#pragma unroll
    for (int y = 0; y < 8; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};

  issue_stage(a, b, kp, kbeg, lds);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int it = 0; it < nk; ++it) {
    v8i fa[8], fb[8];
    read_frags(lds + (it & 1) * STAGEB, fa, fb);
    if (it + 1 < nk) issue_stage(a, b, kp, kbeg + (it + 1) * KS, lds + ((it + 1) & 1) * STAGEB);
    mma_stage(fa, fb, acc);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wr = w >> 1, wc = w & 1;
  const int row0 = tm * TILE + wr * 128, col0 = tn * TILE + wc * 128;
  // row maxima: lane holds rows 4*(lane>>4)+j of column (lane & 15)
#pragma unroll
  for (int x = 0; x < 8; ++x)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float v = acc[x][0][j];
#pragma unroll
      for (int y = 1; y < 8; ++y) v = fmaxf(v, acc[x][y][j]);
      v = fmaxf(v, __shfl_xor(v, 1));
      v = fmaxf(v, __shfl_xor(v, 2));
      v = fmaxf(v, __shfl_xor(v, 4));
      v = fmaxf(v, __shfl_xor(v, 8));
      if ((lane & 15) == 0)
        atomicMax(Rmax + (size_t)slab * mp + row0 + x * 16 + 4 * (lane >> 4) + j, (uint32_t)v);
    }
#pragma unroll
  for (int y = 0; y < 8; ++y) {
    float v = acc[0][y][0];
#pragma unroll
    for (int x = 0; x < 8; ++x)
#pragma unroll
      for (int j = 0; j < 4; ++j) v = fmaxf(v, acc[x][y][j]);
    v = fmaxf(v, __shfl_xor(v, 16));
    v = fmaxf(v, __shfl_xor(v, 32));
    if (lane < 16) atomicMax(Kmax + (size_t)slab * np + col0 + y * 16 + lane, (uint32_t)v);
  }
}

// ------------------------------------------------------------- residue GEMM
// grid: (tiles, r).  One modulus per workgroup over K in [kbeg, kend).
__global__ void __launch_bounds__(256, 1)
k_resgemm(Oz2Const c, const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, int mp,
          int np, int kp, int kbeg, int kend, int accumulate, int16_t* __restrict__ res) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int ntm = mp / TILE;
  const int tile = blockIdx.x, mi = blockIdx.y;
  const int tm = tile % ntm, tn = tile / ntm;
  const int m = c.m[mi], s = c.sq[mi], pb = c.pbase[mi];
  const float inv = c.finv[mi];
  const size_t psA = (size_t)mp * kp, psB = (size_t)np * kp;
  const uint8_t* a0 = PA + (size_t)pb * psA + (size_t)tm * TILE * kp;
  const uint8_t* b0 = PB + (size_t)pb * psB + (size_t)tn * TILE * kp;
  // pairs of planes (A plane, B plane) and chain boundaries:
  //   square:    q=0 (1,0), q=1 (0,1)  -> chain 0 ends, x rho0 (= s)
  //              q=2 (0,0)             -> final, x 1
  //   nonsquare: q=0 (1,1)             -> chain 0 ends, x rho0 (= -16)
  //              q=1 (0,0)             -> chain 1 ends, x rho1 (= -15/16)
  //              q=2 (2,2)             -> final, x 16
  auto planeA = [s](int q) { return s ? (q == 0 ? 1 : 0) : (q == 0 ? 1 : (q == 1 ? 0 : 2)); };
  auto planeB = [s](int q) { return s ? (q == 1 ? 1 : 0) : (q == 0 ? 1 : (q == 1 ? 0 : 2)); };
  const int nk = (kend - kbeg) / KS;

  v4f acc[8][8];
#pragma unroll
  for (int x = 0; x < 8; ++x)
#pragma unroll
    for (int y = 0; y < 8; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};

  issue_stage(a0 + (size_t)planeA(0) * psA, b0 + (size_t)planeB(0) * psB, kp, kbeg, lds);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int q = 0; q < 3; ++q) {
    for (int ks = 0; ks < nk; ++ks) {
      v8i fa[8], fb[8];
      read_frags(lds + ((q * nk + ks) & 1) * STAGEB, fa, fb);
      const int qn = (ks + 1 == nk) ? q + 1 : q, ksn = (ks + 1 == nk) ? 0 : ks + 1;
      if (qn < 3)
        issue_stage(a0 + (size_t)planeA(qn) * psA, b0 + (size_t)planeB(qn) * psB, kp,
                    kbeg + ksn * KS, lds + ((q * nk + ks + 1) & 1) * STAGEB);
      mma_stage(fa, fb, acc);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    }
    if (s ? (q == 1) : (q < 2)) {
      // chain transition: acc <- (acc * rho) reduced mod m, |result| <= m/2 + 2
      const int rho = (q == 0 || s) ? c.rho0[mi] : c.rho1[mi];
#pragma unroll
      for (int x = 0; x < 8; ++x) {
#pragma unroll
        for (int y = 0; y < 8; ++y)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int v = (int)acc[x][y][j];
            acc[x][y][j] = (float)oz2_red(oz2_red(v, m, inv) * rho, m, inv);
          }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }

  // final epilogue: centred residue of fin * acc (+ previous slab's residue)
  const int fin = c.fin[mi];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int16_t* dst = res + (size_t)mi * mp * np + (size_t)tile * (TILE * TILE) + (size_t)w * 16384 +
                 lane * 4;
#pragma unroll
  for (int x = 0; x < 8; ++x)
#pragma unroll
    for (int y = 0; y < 8; ++y) {
      int r4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int v = (int)acc[x][y][j];
        if (fin != 1) v = oz2_red(v, m, inv) * fin;
        r4[j] = oz2_centre(v, m, inv);
      }
      uint2* p = reinterpret_cast<uint2*>(dst + (x * 8 + y) * 256);
      if (accumulate) {
        uint2 o = *p;
        int o4[4] = {(int)(int16_t)(o.x & 0xFFFF), (int)(int16_t)(o.x >> 16),
                     (int)(int16_t)(o.y & 0xFFFF), (int)(int16_t)(o.y >> 16)};
#pragma unroll
        for (int j = 0; j < 4; ++j) r4[j] = oz2_centre(r4[j] + o4[j], m, inv);
      }
      uint2 o;
      o.x = ((uint32_t)r4[0] & 0xFFFFu) | ((uint32_t)r4[1] << 16);
      o.y = ((uint32_t)r4[2] & 0xFFFFu) | ((uint32_t)r4[3] << 16);
      *p = o;
    }
}

bool g_attr_done = false;

hipError_t set_attrs() {
  if (g_attr_done) return hipSuccess;
  hipError_t e = hipFuncSetAttribute((const void*)k_codegemm,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)k_resgemm, hipFuncAttributeMaxDynamicSharedMemorySize,
                          LDS_BYTES);
  if (e != hipSuccess) return e;
  g_attr_done = true;
  return hipSuccess;
}

}  // namespace

hipError_t oz2_launch_codegemm(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, hipStream_t s) {
  hipError_t e = set_attrs();
  if (e != hipSuccess) return e;
  dim3 grid((d.mp / TILE) * (d.np / TILE), d.cslabs);
  hipLaunchKernelGGL(k_codegemm, grid, dim3(256), LDS_BYTES, s, ws + L.codesA, ws + L.codesB, d.mp,
                     d.np, d.kp, d.k, (uint32_t*)(ws + L.Rmax), (uint32_t*)(ws + L.Kmax));
  return hipGetLastError();
}

hipError_t oz2_launch_resgemm(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                              uint8_t* ws, hipStream_t s) {
  hipError_t e = set_attrs();
  if (e != hipSuccess) return e;
  dim3 grid((d.mp / TILE) * (d.np / TILE), c.r);
  for (int kb = 0, sl = 0; kb < d.kp; kb += OZ2_KSLAB, ++sl) {
    int ke = kb + OZ2_KSLAB < d.kp ? kb + OZ2_KSLAB : d.kp;
    hipLaunchKernelGGL(k_resgemm, grid, dim3(256), LDS_BYTES, s, c, ws + L.planesA, ws + L.planesB,
                       d.mp, d.np, d.kp, kb, ke, sl > 0 ? 1 : 0, (int16_t*)(ws + L.res));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
