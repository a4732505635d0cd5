// The residue GEMMs of Phase 2 and the reconstruction of Phase 3 in one
// kernel, for r <= 12 moduli and k within one exact FP32 slab: the fused
// reconstruction epilogue.  The staged path writes every output's r residues
// to HBM (1.5 r bytes per output) and reads them back in the reconstruction;
// here a workgroup walks all r moduli of its 128 x 128 output tile, keeps
// each output's residues packed in registers, and at the end forms the exact
// CRT integer (the reconstruction's own routine), rounds it once with the
// shift -(s_i + t_j) (Eq. (scale) undone), and writes C (C_in + C with
// OZ2_ACCUMULATE).  Per output and modulus the residue is a representative
// x with |x| <= m/2 + 32, stored as x + floor(m/2) + 32 in a bit field of
// ceil(log2(m + 65)) bits; the twelve fields of r = 12 take 123 of the four
// 32-bit words (assigned at compile time, first fit by decreasing width).
//
// Per modulus the three E4M3 plane products of Eq. (sq-shortcut) / Eq. (kar)
// run as chains on one accumulator set, exactly as in the staged residue
// GEMM (every partial sum an integer <= 2^24, Eq. (accum-exact)); operands
// stream through a 4-deep LDS ring (16 KiB per K = 64 stage) filled by
// global_load_lds_dwordx4 three stages ahead, one barrier per stage.
// 8 waves (2 per SIMD); wave w owns rows 32 (w/2) .. +31 and columns
// 64 (w%2) .. +63 of the tile: one A fragment and two B fragments per stage,
// two v_mfma_f32_32x32x64_f8f6f4, 32 outputs per lane.
#include "oz2_device.h"

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) uint8_t lds_u8;

constexpr int FT = 128;            // output tile (rows and columns)
constexpr int KS = OZ2_KBLK;       // k bytes per stage
constexpr int FOPB = FT * KS;      // 8 KiB per operand per stage
constexpr int FSTB = 2 * FOPB;     // 16 KiB per stage
constexpr int FNB = 4;             // ring depth
constexpr int FNT = 512;           // threads (8 waves)
constexpr int TRP = 33;            // doubles per transposed column (32 + 1: banks spread)
constexpr int FTR = 8 * 32 * TRP * 8;    // the epilogue's transposition (66 KiB), over the ring
// the fourth word of every output's packed residues lives in LDS (64 KiB:
// [wave][output][lane]); the other three stay in registers
constexpr int FPK3 = FTR;
static_assert(FNB * FSTB <= FTR, "the ring lies inside the transposition's space");
constexpr int FLDS = FPK3 + 8 * 32 * 64 * 4;

__device__ __forceinline__ void bar() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}
__device__ __forceinline__ void wait_lgkm0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// XOR chunk swizzle of LDS row r (conflict-free fragment reads for 16 rows)
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 3) ^ ((r >> 3) & 1); }
// global_load_lds_dwordx4: lane L's 16 bytes land at M0 + 16 L
__device__ __forceinline__ void dma16(const uint8_t* sbase, uint32_t voff, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 sc1" ::"v"(voff), "s"(sbase),
               "s"(m0)
               : "memory");
}
// planes of product q: square (1,0) (0,1) | (0,0); nonsquare (1,1) | (0,0) | (2,2)
__device__ __forceinline__ int planeA(int s, int q) {
  return s ? (q == 0 ? 1 : 0) : (q == 0 ? 1 : (q == 1 ? 0 : 2));
}
__device__ __forceinline__ int planeB(int s, int q) {
  return s ? (q == 1 ? 1 : 0) : (q == 0 ? 1 : (q == 1 ? 0 : 2));
}

// ---- the bit fields of the packed residues, per moduli count R <= 12 ----
// The moduli of R are the R largest of the pool, in ascending order (the
// host checks the plan's constants against this list before launching).
constexpr int kPoolDesc[OZ2_MAXR] = {1089, 1024, 961, 841, 625, 529, 511, 509,
                                     503,  499,  491, 487, 481, 479, 467, 463};
constexpr int bitlen(int v) {
  int b = 0;
  while (v) {
    ++b;
    v >>= 1;
  }
  return b;
}
struct Pack {
  int word[12], shift[12], fits;
};
template <int R>
constexpr Pack make_pack() {
  Pack p{};
  int used[4] = {0, 0, 0, 0};
  p.fits = 1;
  for (int i = R - 1; i >= 0; --i) {   // modulus i is kPoolDesc[R - 1 - i]; widest first
    const int b = bitlen(kPoolDesc[R - 1 - i] + 64);
    int wd = -1;
    for (int q = 0; q < 4 && wd < 0; ++q)
      if (used[q] + b <= 32) wd = q;
    if (wd < 0) {
      p.fits = 0;
      wd = 0;
    }
    p.word[i] = wd;
    p.shift[i] = used[wd];
    used[wd] += b;
  }
  return p;
}
template <int R>
struct Packing {
  static constexpr Pack p = make_pack<R>();
  static_assert(p.fits, "the packed residues of r <= 12 moduli fit four 32-bit words");
};
template <int R>
__device__ __forceinline__ uint32_t field_mask(int i) {
  return (1u << bitlen(kPoolDesc[R - 1 - i] + 64)) - 1u;
}

// Tile of block b: each XCD (blocks dispatched round-robin over 8) gets a
// 4 x 8 group of tiles per 256 blocks when the grid allows it.
__device__ __forceinline__ int ftile_of(int b, int ntm, int ntn) {
  if ((ntm % 4) || (ntn % 8) || ((ntm * ntn) % 256)) return b;
  const int xcd = b & 7, slot = b >> 3;
  const int grp = slot >> 5, in = slot & 31;
  const int gid = grp * 8 + xcd, ngx = ntm / 4;
  const int gm = gid % ngx, gn = gid / ngx;
  return (gm * 4 + (in & 3)) + (gn * 8 + (in >> 2)) * ntm;
}

// The operand stream of one workgroup: stages of product q of modulus mi at
// k-block kb, walked in order (kb fastest, then q, then mi).
struct FStream {
  const uint8_t* a0;    // planes of A at the tile's first row, k-block 0
  const uint8_t* b0;
  size_t psA, psB, kbA, kbB;
  int nk, T;
  const uint8_t* pa;    // current stage's blocks
  const uint8_t* pb;
  int left, q, mi;
  uint32_t vo, mw;      // lane offset in the wave's 1 KiB block; w * 1 KiB
};

__device__ __forceinline__ void fs_product(const Oz2Const& c, FStream& f) {
  const int s = c.sq[f.mi], p0 = c.pbase[f.mi];
  f.pa = f.a0 + (size_t)(p0 + planeA(s, f.q)) * f.psA;
  f.pb = f.b0 + (size_t)(p0 + planeB(s, f.q)) * f.psB;
}

// wave w's share of one stage: A block w and B block w (16 rows each)
__device__ __forceinline__ void fs_issue(const Oz2Const& c, FStream& f, uint32_t slot) {
  dma16(f.pa, f.vo, slot + f.mw);
  dma16(f.pb, f.vo, slot + FOPB + f.mw);
  f.pa += f.kbA;
  f.pb += f.kbB;
  if (--f.left == 0) {
    f.left = f.nk;
    if (++f.q == 3) {
      f.q = 0;
      ++f.mi;
    }
    if (f.mi < c.r) fs_product(c, f);
  }
}

__device__ __forceinline__ v8i ldfrag(const uint8_t* p, int o0, int o1) {
  const uint4 lo = *reinterpret_cast<const uint4*>(p + o0);
  const uint4 hi = *reinterpret_cast<const uint4*>(p + o1);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// stages [t0, t0 + n): wait for stage t, barrier, refill the slot of stage
// t - 1 with stage t + 3, then the stage's fragments and MFMAs
__device__ __forceinline__ void fs_run(const Oz2Const& c, FStream& f, const uint8_t* LB,
                                       uint32_t lds0, int t0, int n, v16f (&acc)[2]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wr = w >> 1, wc = w & 1;
  const int h = lane >> 5, sw = swz(lane & 31);
  const int o0 = 16 * ((2 * h) ^ sw), o1 = 16 * ((2 * h + 1) ^ sw);
  const int T = f.T;
  for (int t = t0; t < t0 + n; ++t) {
    // this wave's DMA of stage t has landed once at most those of the
    // stages after it (up to t + 2, two instructions each) are in flight
    if (t + 2 < T) wait_vm<4>();
    else if (t + 1 < T) wait_vm<2>();
    else wait_vm<0>();
    bar();
    if (t + 3 < T) fs_issue(c, f, lds0 + ((t + 3) & 3) * FSTB);
    const uint8_t* st = LB + (t & 3) * FSTB;
    const v8i fa = ldfrag(st + (wr * 32 + (lane & 31)) * KS, o0, o1);
    const v8i fb0 = ldfrag(st + FOPB + (wc * 64 + (lane & 31)) * KS, o0, o1);
    const v8i fb1 = ldfrag(st + FOPB + (wc * 64 + 32 + (lane & 31)) * KS, o0, o1);
    wait_lgkm0();
    acc[0] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa, fb0, acc[0], 0, 0, 0, 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa, fb1, acc[1], 0, 0, 0, 0, 0, 0);
  }
}

__device__ __forceinline__ void chain_reduce(v16f (&acc)[2], float inv, float fm, float rho) {
#pragma unroll
  for (int y = 0; y < 2; ++y)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float v = acc[y][e];
      acc[y][e] = __builtin_fmaf(-rintf(v * inv), fm, v) * rho;
    }
}
__device__ __forceinline__ void chain_scale(v16f (&acc)[2], float f) {
#pragma unroll
  for (int y = 0; y < 2; ++y) acc[y] *= f;
}

// the modulus's residues (fin * acc reduced: |x| <= m/2 + 32) into their bit
// fields of word W (words 0-2 in registers, word 3 in the lane's LDS slots)
template <int W>
__device__ __forceinline__ void pack_into(uint32_t (&pk)[3][32], uint32_t* pk3,
                                          const v16f (&acc)[2], float fin, float fm, float inv,
                                          float off, int shift) {
#pragma unroll
  for (int y = 0; y < 2; ++y)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float v = acc[y][e] * fin;
      const float x = __builtin_fmaf(-rintf(v * inv), fm, v) + off;
      const uint32_t fld = (uint32_t)(int)x << shift;
      if constexpr (W < 3) pk[W][16 * y + e] |= fld;
      else pk3[(16 * y + e) * 64] |= fld;
    }
}

template <int R>
__global__ void __launch_bounds__(FNT, 1)
k_resgemm_crt(Oz2Const c, Oz2Dims d, const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB,
              int cheap, const int32_t* __restrict__ sA, const int32_t* __restrict__ tB,
              const uint32_t* __restrict__ fA, const uint32_t* __restrict__ fB, double* C,
              int ldc) {
  extern __shared__ __attribute__((aligned(16))) uint8_t LB[];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u8*)LB;
  const int ntm = d.mp / FT, ntn = d.np / FT;
  const int tile = ftile_of(blockIdx.x, ntm, ntn);
  const int tm = tile % ntm, tn = tile / ntm;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  FStream f;
  f.psA = (size_t)d.mp * d.kp;
  f.psB = (size_t)d.np * d.kp;
  f.kbA = (size_t)d.mp * KS;
  f.kbB = (size_t)d.np * KS;
  f.a0 = PA + (size_t)tm * FT * KS;
  f.b0 = PB + (size_t)tn * FT * KS;
  f.nk = d.kp / KS;
  f.T = 3 * f.nk * R;
  {
    const int wu = __builtin_amdgcn_readfirstlane(w);
    const int rb = lane >> 2;
    f.vo = (uint32_t)(rb * KS + 16 * ((lane & 3) ^ swz(rb))) + (uint32_t)wu * 1024u;
    f.mw = (uint32_t)wu * 1024u;
  }
  f.left = f.nk;
  f.q = 0;
  f.mi = 0;
  fs_product(c, f);
#pragma unroll
  for (int t = 0; t < FNB - 1; ++t)
    if (t < f.T) fs_issue(c, f, lds0 + t * FSTB);

  uint32_t pk[3][32];
#pragma unroll
  for (int q = 0; q < 3; ++q)
#pragma unroll
    for (int o = 0; o < 32; ++o) pk[q][o] = 0u;
  uint32_t* pk3 = reinterpret_cast<uint32_t*>(LB + FPK3) + (size_t)w * 32 * 64 + lane;
#pragma unroll
  for (int o = 0; o < 32; ++o) pk3[o * 64] = 0u;
  const int nk = f.nk;
  int it = 0;
  // unrolled: the modulus's field position (and whether it is square: the
  // six largest moduli are) are compile-time constants in each copy
#pragma unroll
  for (int mi = 0; mi < R; ++mi) {
    const int m = c.m[mi], s = mi >= R - 6 ? c.sq[mi] : 0;
    const float fm = (float)m, inv = c.finv[mi];
    v16f acc[2];
    acc[0] = v16f{0.f};
    acc[1] = v16f{0.f};
    if (s) {
      fs_run(c, f, LB, lds0, it, 2 * nk, acc);
      if (cheap & 1) chain_scale(acc, (float)s);
      else chain_reduce(acc, inv, fm, (float)s);
      fs_run(c, f, LB, lds0, it + 2 * nk, nk, acc);
    } else {
      fs_run(c, f, LB, lds0, it, nk, acc);
      if (cheap & 2) chain_scale(acc, -16.0f);
      else chain_reduce(acc, inv, fm, (float)c.rho0[mi]);
      fs_run(c, f, LB, lds0, it + nk, nk, acc);
      chain_reduce(acc, inv, fm, (float)c.rho1[mi]);
      fs_run(c, f, LB, lds0, it + 2 * nk, nk, acc);
    }
    it += 3 * nk;
    const float fin = (float)c.fin[mi], off = (float)(m / 2 + 32);
    constexpr Pack P = Packing<R>::p;
    const int sh = P.shift[mi];
    switch (P.word[mi]) {
      case 0: pack_into<0>(pk, pk3, acc, fin, fm, inv, off, sh); break;
      case 1: pack_into<1>(pk, pk3, acc, fin, fm, inv, off, sh); break;
      case 2: pack_into<2>(pk, pk3, acc, fin, fm, inv, off, sh); break;
      default: pack_into<3>(pk, pk3, acc, fin, fm, inv, off, sh); break;
    }
  }
  bar();   // every wave is past its last fragment reads: the ring is free

  // CRT, rounding, and the store through a per-wave 32 x 32 transposition
  // (lane L holds column L%32, rows 8(e/4) + 4(L/32) + e%4 of each 32 x 32
  // block; the store writes 32 consecutive rows of a column per half-wave)
  double* T = reinterpret_cast<double*>(LB) + (size_t)w * 32 * TRP;
  const int wr = w >> 1, wc = w & 1;
  const int row0 = tm * FT + wr * 32, cl = lane & 31;
  const bool accum = (d.flags & 1u) != 0;   // OZ2_ACCUMULATE
  const bool nofb = (d.flags & 8u) != 0;    // OZ2_NO_FALLBACK
  const bool force = (d.flags & 16u) != 0;  // OZ2_FORCE_FALLBACK
  // every per-row and per-column value the half needs is loaded before its
  // CRT work, with no divergent branch around a load, so that the loads'
  // latency is paid once and hidden behind the CRT (the scale and flag
  // arrays hold mp and np entries: the tile's padded rows and columns are in
  // bounds; C_in's address is clamped to the matrix, and what is read for a
  // padded or flagged output is never stored)
  const int srow = row0 + (lane & 31);     // the store layout's row of this lane
  const int crow = srow < d.m ? srow : d.m - 1;
  const uint32_t fa = fA[srow];
  const bool rok = srow < d.m && (nofb || !(force || (fa & (OZ2_T1 | OZ2_T2))));
#pragma unroll
  for (int y = 0; y < 2; ++y) {
    const int col0 = tn * FT + wc * 64 + 32 * y;
    const int tj = tB[col0 + cl];
    int si[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) si[e] = sA[row0 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)];
    // the store layout: column col0 + 2 j + lane / 32 of row srow
    uint32_t okm = 0;
    double cin[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int cj = col0 + 2 * j + (lane >> 5);
      const uint32_t fb = fB[cj];
      okm |= (rok && cj < d.n && (nofb || !(fb & (OZ2_T1 | OZ2_T2)))) ? 1u << j : 0u;
      cin[j] = 0.0;
      if (accum)
        cin[j] = __builtin_nontemporal_load(C + (size_t)(cj < d.n ? cj : d.n - 1) * ldc + crow);
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int rr = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      double x[R];
      constexpr Pack P = Packing<R>::p;
      const uint32_t w3 = pk3[(16 * y + e) * 64];
#pragma unroll
      for (int i = 0; i < R; ++i) {
        const uint32_t wd = P.word[i] == 3 ? w3 : pk[P.word[i] < 3 ? P.word[i] : 0][16 * y + e];
        const uint32_t fld = (wd >> P.shift[i]) & field_mask<R>(i);
        x[i] = (double)(int)fld - (double)(kPoolDesc[R - 1 - i] / 2 + 32);
      }
      double S[3];
      crt38_sum<R, 3>(c, x, S);
      T[cl * TRP + rr] = round38<3>(S, si[e] + tj);
      // one output at a time: interleaving several CRTs would need more
      // registers than the packed residues leave
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    const int rr = lane & 31;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int cc = 2 * j + (lane >> 5), cj = col0 + cc;
      if ((okm >> j) & 1u) {
        const double v = T[cc * TRP + rr];
        __builtin_nontemporal_store(accum ? cin[j] + v : v, C + (size_t)cj * ldc + srow);
      }
    }
    __syncthreads();
  }
}

template <int R>
hipError_t launch_fused_r(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                          double* C, int ldc, hipStream_t s) {
  // the first chain transition may skip its reduction when every modulus of
  // a kind has k <= kcheap
  bool sq_cheap = true, ns_cheap = true;
  for (int i = 0; i < c.r; ++i) {
    const bool ok = d.kp <= c.kcheap[i];
    if (c.sq[i]) sq_cheap = sq_cheap && ok;
    else ns_cheap = ns_cheap && ok;
  }
  const int cheap = (sq_cheap ? 1 : 0) | (ns_cheap ? 2 : 0);
  (void)hipFuncSetAttribute((const void*)k_resgemm_crt<R>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, FLDS);
  const unsigned tiles = (unsigned)((d.mp / FT) * (d.np / FT));
  hipLaunchKernelGGL(k_resgemm_crt<R>, dim3(tiles), dim3(FNT), FLDS, s, c, d, ws + L.planesA,
                     ws + L.planesB, cheap, (const int32_t*)(ws + L.sA),
                     (const int32_t*)(ws + L.tB), (const uint32_t*)(ws + L.flagsA),
                     (const uint32_t*)(ws + L.flagsB), C, ldc);
  return hipGetLastError();
}

}  // namespace

hipError_t oz2_launch_fused(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                            double* C, int ldc, hipStream_t s) {
  if (d.kp > OZ2_KSLAB || c.r > 12) return hipErrorInvalidValue;
  for (int i = 0; i < c.r; ++i)
    if (c.m[i] != kPoolDesc[c.r - 1 - i]) return hipErrorInvalidValue;
  switch (c.r) {
    case 8: return launch_fused_r<8>(d, L, c, ws, C, ldc, s);
    case 9: return launch_fused_r<9>(d, L, c, ws, C, ldc, s);
    case 10: return launch_fused_r<10>(d, L, c, ws, C, ldc, s);
    case 11: return launch_fused_r<11>(d, L, c, ws, C, ldc, s);
    case 12: return launch_fused_r<12>(d, L, c, ws, C, ldc, s);
    default: return hipErrorInvalidValue;
  }
}
