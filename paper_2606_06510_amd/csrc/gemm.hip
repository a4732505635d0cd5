// FP8 MFMA GEMMs of Alg. 1 on gfx950 (v_mfma_f32_32x32x64_f8f6f4, E4M3 x E4M3,
// FP32 accumulation):
//
//  * the max-magnitude pass ("+1" of alpha = 3r+1): G' = codesA * codesB^T,
//    epilogue = row / column maxima (integer atomics); G' is never stored;
//  * Phase 2, Eq. (modgemm): per modulus, the three E4M3 plane products of
//    Eq. (sq-shortcut) (square m = s^2: d1e0 + d0e1 with coefficient s, then
//    d0e0 with coefficient 1) or Eq. (kar) with b = 4 (nonsquare: d1e1 with
//    240, d0e0 with -15, (d0+d1)(e0+e1) with 16), accumulated exactly in FP32
//    (Eq. (accum-exact): every partial sum is an integer of magnitude
//    <= 2^24 for k <= 32768), then reduced mod m (to a representative of
//    magnitude <= m/2 + 32; see the epilogue).
//
// Design.  One workgroup (8 waves, 2 per SIMD) owns a 256x256 output tile;
// wave w owns 128x64 of it (4x2 MFMA tiles of 32x32, 128 FP32 accumulators
// per lane), so while one wave of a SIMD waits at a barrier or runs a chain
// transition the other keeps the matrix unit busy.  Operands are K-blocked
// E4M3 planes ([k/64][rows][64 B]): one K=64 stage of a 256-row tile is one
// contiguous 16 KiB block.  Stages stream into a 4-deep LDS ring (32 KiB per
// stage) through global_load_lds_dwordx4 (issued by inline asm, so every
// wait on it is explicit: s_waitcnt vmcnt + s_barrier), three stages ahead,
// with an XOR swizzle of the 16-byte chunks (row bits 1..3) that keeps the
// fragment reads bank-conflict free.  The three products of a modulus run as
// sequential "chains" on ONE accumulator set: where the coefficient changes,
// the exact integer accumulator is reduced mod m and multiplied by
// c_this / c_next (mod m), so the next product continues the same residue.
#include <algorithm>

#include "oz2_internal.h"

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) uint8_t lds_u8;

constexpr int TILE = OZ2_TILE;   // 256
constexpr int KS = OZ2_KBLK;     // 64 k bytes per stage
constexpr int OPB = TILE * KS;   // 16 KiB per operand per stage
constexpr int STB = 2 * OPB;     // 32 KiB per stage
constexpr int NB = 4;            // ring depth
constexpr int NT = 512;          // threads per workgroup

// s_barrier pinned in the instruction stream: the scheduler moves nothing
// (not even register-only MFMAs) across it, so the phases below stay phases
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

// chunk swizzle of LDS row r: conflict free for 16 consecutive rows
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 3) ^ ((r >> 3) & 1); }

// global_load_lds_dwordx4: lane L's 16 bytes land at M0 + 16 L.  The sc1
// cache policy (streaming operands with no reuse inside the CU's vector L1)
// measured 10-12% faster than the default policy on the 4096^3 residue GEMMs.
__device__ __forceinline__ void dma16(const uint8_t* sbase, uint32_t voff, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 sc1" ::"v"(voff), "s"(sbase),
               "s"(m0)
               : "memory");
}

// Per-wave DMA stream over a sequence of plane products.  The code GEMM is a
// single product; a residue-GEMM workgroup walks moduli mi0 .. mi1-1 of its
// tile, three products each, as one continuous stream (the next modulus's
// first stages load while the previous one's epilogue runs).  All of it is
// uniform (SGPRs): a stage costs four DMA instructions and a few scalar adds.
// planes of product q: square  (1,0) (0,1) | (0,0);  nonsquare (1,1) | (0,0) | (2,2)
__device__ __forceinline__ int planeA(int s, int q) {
  return s ? (q == 0 ? 1 : 0) : (q == 0 ? 1 : (q == 1 ? 0 : 2));
}
__device__ __forceinline__ int planeB(int s, int q) {
  return s ? (q == 1 ? 1 : 0) : (q == 0 ? 1 : (q == 1 ? 0 : 2));
}

struct Ctx {
  const uint8_t* a0;      // plane 0 (the codes) at the tile's first row, k-block kbeg
  const uint8_t* b0;
  size_t psA, psB;        // plane strides
  size_t kbA, kbB;        // k-block strides (padded rows * 64)
  int nk, T;              // stages per product, total stages
  int mi1;                // residue GEMM: one past the workgroup's last modulus
};

struct Dma {
  const uint8_t* pa;
  const uint8_t* pb;
  int left, q, mi;        // stages left in product q of modulus mi
  uint32_t vo0, vo1;      // lane offsets of blocks w and w + 8 (VGPR)
  uint32_t mw;            // w * 1 KiB (uniform)
};

// operand blocks of product q of modulus mi at k-block kbeg
__device__ __forceinline__ void product_ptrs(const Oz2Const* c, const Ctx& x, int mi, int q, Dma& d) {
  const int s = c->sq[mi], p0 = c->pbase[mi];
  d.pa = x.a0 + (size_t)(p0 + planeA(s, q)) * x.psA;
  d.pb = x.b0 + (size_t)(p0 + planeB(s, q)) * x.psB;
}

// One stage = A tile (16 x 1 KiB blocks of 16 rows) + B tile (16 blocks);
// wave w moves blocks w and w + 8 of each.  Lane L writes row 16 blk + L/4,
// physical chunk L%4 = logical chunk ^ swz.
__device__ __forceinline__ Dma dma_init(const Ctx& x) {
  Dma d;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rb = lane >> 2;
  const uint32_t lo = (uint32_t)(rb * KS + 16 * ((lane & 3) ^ swz(rb)));
  d.vo0 = lo + (uint32_t)w * 1024u;
  d.vo1 = d.vo0 + 8u * 1024u;
  d.mw = (uint32_t)w * 1024u;
  d.pa = x.a0;
  d.pb = x.b0;
  d.left = x.nk;
  d.q = 0;
  d.mi = 0;
  return d;
}

// RES: advance through the residue products up to modulus Ctx::mi1 (c = the
// plan constants); otherwise the stream is the single code product (c unused).
template <bool RES>
__device__ __forceinline__ void issue_stage(const Oz2Const* c, const Ctx& x, Dma& d,
                                            uint32_t lbase) {
  dma16(d.pa, d.vo0, lbase + d.mw);
  dma16(d.pa, d.vo1, lbase + d.mw + 8u * 1024u);
  dma16(d.pb, d.vo0, lbase + OPB + d.mw);
  dma16(d.pb, d.vo1, lbase + OPB + d.mw + 8u * 1024u);
  d.pa += x.kbA;
  d.pb += x.kbB;
  if (RES && --d.left == 0) {
    d.left = x.nk;
    if (++d.q == 3) {
      d.q = 0;
      ++d.mi;
    }
    if (d.mi < x.mi1) product_ptrs(c, x, d.mi, d.q, d);
  }
}

__device__ __forceinline__ v8i ldfrag(const uint8_t* p, int o0, int o1) {
  const uint4 lo = *reinterpret_cast<const uint4*>(p + o0);
  const uint4 hi = *reinterpret_cast<const uint4*>(p + o1);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// Fragments of wave w: rows (w>>2)*128 + 32x + lane%32, columns (w&3)*64 + 32y
// + lane%32; lane half h = lane/32 holds k bytes 32h..32h+31.
__device__ __forceinline__ void frags(const uint8_t* st, v8i (&fa)[4], v8i (&fb)[2]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wr = w >> 2, wc = w & 3;
  const int h = lane >> 5, sw = swz(lane & 31);
  const int o0 = 16 * ((2 * h) ^ sw), o1 = 16 * ((2 * h + 1) ^ sw);
  const uint8_t* sa = st + (wr * 128 + (lane & 31)) * KS;
  const uint8_t* sb = st + OPB + (wc * 64 + (lane & 31)) * KS;
#pragma unroll
  for (int x = 0; x < 4; ++x) fa[x] = ldfrag(sa + x * 32 * KS, o0, o1);
#pragma unroll
  for (int y = 0; y < 2; ++y) fb[y] = ldfrag(sb + y * 32 * KS, o0, o1);
}

// Tile of block b.  Blocks are dispatched round-robin over the 8 XCDs (each
// with its own L2); when the grid allows it each XCD gets a 4x8 group of
// tiles per 256-block round (4 A row panels, 8 B column panels).
__device__ __forceinline__ int tile_of(int b, int ntm, int ntn) {
  if ((ntm % 4) || (ntn % 8) || ((ntm * ntn) % 256)) return b;
  const int xcd = b & 7, slot = b >> 3;
  const int grp = slot >> 5, in = slot & 31;
  const int gid = grp * 8 + xcd, ngx = ntm / 4;
  const int gm = gid % ngx, gn = gid / ngx;
  return (gm * 4 + (in & 3)) + (gn * 8 + (in >> 2)) * ntm;
}

// Wait until this wave's DMA share of stage s has landed.  When it waits
// for stage s the wave has issued its shares up to stage min(s + 2, T - 1)
// (four DMA instructions each, returning in order); stages below `landed`
// are known to be in LDS already (the wave drained its loads before the
// epilogue stores that now share its vmcnt).
__device__ __forceinline__ void wait_stage(int s, int T, int landed) {
  if (s >= T || s < landed) return;
  if (s + 2 < T) wait_vm<8>();
  else if (s + 1 < T) wait_vm<4>();
  else wait_vm<0>();
}

// Main loop over stages [it0, it0 + n) of the stage sequence, in two phases
// per stage separated by workgroup barriers:
//   L(t): issue this wave's DMA share of stage t + 3 (ring slot (t+3)%4, last
//         read in L(t-1)), read the fragments of stage t from LDS and wait
//         for them;
//   C(t): the 8 MFMAs of stage t.
// The two waves sharing a SIMD (w and w + 4) run the same sequence one phase
// apart (group g = w / 4; group 1 passes one extra barrier first, group 0 one
// extra barrier last), so while one issues its LDS reads, DMAs, waits and
// chain transitions the other keeps the SIMD's matrix unit busy.  Barrier b
// sees C(t) of group 0 end with L(t) of group 1 (b = 2t + 1) and L(t+1) of
// group 0 end with C(t) of group 1 (b = 2t + 2); stage t + 1 must have landed
// by barrier 2t + 1, the first one before anyone reads it, and the
// fragment reads of slot t%4 are complete by barrier 2t + 1 as well, before
// any wave's L(t+1) may issue the DMA that overwrites it.
template <bool RES>
__device__ __forceinline__ void run_stages(const Oz2Const* c, const Ctx& x, Dma& dm, uint8_t* LB,
                                           uint32_t lds0, int it0, int n, int landed, int g,
                                           v16f (&acc)[4][2]) {
  const int T = x.T;
  for (int it = it0; it < it0 + n; ++it) {
    if (it + 3 < T) issue_stage<RES>(c, x, dm, lds0 + ((it + 3) & 3) * STB);
    v8i fa[4], fb[2];
    frags(LB + (it & 3) * STB, fa, fb);
    wait_lgkm0();
    if (g) wait_stage(it + 1, T, landed);
    bar();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa[i], fb[j], acc[i][j], 0, 0,
                                                                   0, 0, 0, 0);
    if (!g) wait_stage(it + 1, T, landed);
    bar();
  }
}

// Before the loop: every wave issues its shares of stages 0..2, stage 0 is
// waited for by all, then group 1 takes its one-phase offset.
template <bool RES>
__device__ __forceinline__ void prologue(const Oz2Const* c, const Ctx& x, Dma& dm, uint32_t lds0,
                                         int g) {
#pragma unroll
  for (int t = 0; t < NB - 1; ++t)
    if (t < x.T) issue_stage<RES>(c, x, dm, lds0 + t * STB);
  wait_stage(0, x.T, 0);
  bar();
  if (g) bar();
}

// One step of a halving max-butterfly across lanes L and L^B: of the first N
// entries of u, lane L keeps the half selected by bit B of L (upper when set),
// maximised with the partner's copy of that half, in u[0 .. N/2).
template <int N, int B>
__device__ __forceinline__ void halve(float (&u)[64], int lane) {
  const bool up = (lane & B) != 0;
#pragma unroll
  for (int k = 0; k < N / 2; ++k) {
    const float keep = up ? u[k + N / 2] : u[k];
    const float send = up ? u[k] : u[k + N / 2];
    u[k] = fmaxf(keep, __shfl_xor(send, B));
  }
}

// ------------------------------------------------------------- code GEMM
// grid: (tiles tbase .. tbase + gridDim.x - 1, code slabs).
// G'[i][j] <= 256 * 65536 = 2^24: exact in FP32.
__global__ void __launch_bounds__(NT, 1)
k_codegemm(const uint8_t* __restrict__ cA, const uint8_t* __restrict__ cB, int mp, int np,
           int kp, uint32_t* Rmax, uint32_t* Kmax, int tbase) {
  __shared__ __attribute__((aligned(16))) uint8_t LB[NB * STB];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u8*)LB;
  const int ntm = mp / TILE, ntn = np / TILE;
  const int tile = tile_of(tbase + blockIdx.x, ntm, ntn), slab = blockIdx.y;
  const int tm = tile % ntm, tn = tile / ntm;
  const int kbeg = slab * OZ2_CSLAB, kend = min(kp, kbeg + OZ2_CSLAB);
  Ctx x;
  x.kbA = (size_t)mp * KS;
  x.kbB = (size_t)np * KS;
  x.a0 = cA + (size_t)tm * TILE * KS + (size_t)(kbeg / KS) * x.kbA;
  x.b0 = cB + (size_t)tn * TILE * KS + (size_t)(kbeg / KS) * x.kbB;
  x.psA = x.psB = 0;
  x.nk = (kend - kbeg) / KS;
  x.T = x.nk;
  x.mi1 = 0;
  Dma dm = dma_init(x);
  v16f acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v16f{0.f};
  const int g = __builtin_amdgcn_readfirstlane(threadIdx.x >> 8);
  prologue<false>(nullptr, x, dm, lds0, g);
  run_stages<false>(nullptr, x, dm, LB, lds0, 0, x.T, 0, g, acc);
  if (!g) bar();

  // Row and column maxima of G'.  Lane L holds rows 32i + 8(e/4) + 4(L/32) +
  // e%4 (of the wave's 128) in column 32j + L%32 (of its 64).
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wr = w >> 2, wc = w & 3;
  float u[64];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) u[16 * i + e] = fmaxf(acc[i][0][e], acc[i][1][e]);
  // halving butterfly over the 32 lanes of each half: lane L keeps entries
  // 2(L%32) and 2(L%32) + 1 of u, maximised over its half
  halve<64, 16>(u, lane);
  halve<32, 8>(u, lane);
  halve<16, 4>(u, lane);
  halve<8, 2>(u, lane);
  halve<4, 1>(u, lane);
  float cmax[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    float v = acc[0][j][0];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) v = fmaxf(v, acc[i][j][e]);
    cmax[j] = fmaxf(v, __shfl_xor(v, 32));   // column 32j + L%32 over the wave's rows
  }
  // combine the 4 waves sharing rows and the 2 sharing columns in LDS (the
  // ring is free once every wave is past its last stage), then one atomic per
  // row and per column of the tile
  float* red = reinterpret_cast<float*>(LB);   // [wr][wc][128] row maxima
  float* cred = red + 1024;                    // [wr][wc][64] column maxima
  bar();
  const int h = lane >> 5, q = lane & 31;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int ie = 2 * q + t, i = ie >> 4, e = ie & 15;
    red[(wr * 4 + wc) * 128 + 32 * i + 8 * (e >> 2) + 4 * h + (e & 3)] = u[t];
  }
  if (lane < 32) {
    cred[(wr * 4 + wc) * 64 + lane] = cmax[0];
    cred[(wr * 4 + wc) * 64 + 32 + lane] = cmax[1];
  }
  __syncthreads();
  const int t = threadIdx.x;
  if (t < 256) {
    const int r = t >> 7, row = t & 127;
    const float* p = red + r * 512 + row;
    const float v = fmaxf(fmaxf(p[0], p[128]), fmaxf(p[256], p[384]));
    atomicMax(Rmax + (size_t)slab * mp + tm * TILE + t, (uint32_t)v);
  } else {
    const int col = t - 256, c4 = col >> 6, cc = col & 63;
    const float v = fmaxf(cred[c4 * 64 + cc], cred[(4 + c4) * 64 + cc]);
    atomicMax(Kmax + (size_t)slab * np + tn * TILE + col, (uint32_t)v);
  }
}

// Chain transitions: acc <- (acc - m rint(acc/m)) * rho.  The reduced value
// has magnitude <= m/2 + 3 (the fp32 quotient estimate is within 1 of the
// exact one), so |acc * rho| < 2^18 and the next product keeps every partial
// sum below 2^24.  Square moduli: the two cross products share one chain
// (their sum is at most 512 k_slab = 2^24), then x s before d0e0.
// Nonsquare: d1e1, x rho0 = 240/(-15), d0e0, x rho1 = -15/16,
// (d0+d1)(e0+e1).
__device__ __forceinline__ void chain_reduce(v16f (&acc)[4][2], float inv, float fm, float rho) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float v = acc[i][j][e];
        acc[i][j][e] = __builtin_fmaf(-rintf(v * inv), fm, v) * rho;
      }
}
// the same transition without the reduction, for chains short enough that
// the unreduced product stays exact (k <= kcheap)
__device__ __forceinline__ void chain_scale(v16f (&acc)[4][2], float f) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] *= f;
}

// Residue-GEMM epilogue: a representative of fin * acc (+ the previous
// slab's) mod m, in fp32 throughout.  acc is an integer with |acc| <= 2^24
// and fin is 1 or 16, so v = fin * acc is exact.  v * RN(1/m) is within
// 2 * 2^-24 |v| / m <= 32 / m of v / m (the relative errors of RN(1/m) and of
// the product), so x = v - m rint(.) is an exact integer of magnitude
// <= m/2 + 32.  The reconstruction's exact CRT sum takes any representative
// of that size (the canonical centring is left to the diagnostic residue
// query).  With a previous slab, the sum (|.| <= m + 64) is reduced once
// more: its quotient estimate is then within 2^-22 of the exact one, so the
// result lies in [-m/2, m/2].
// Stored: u = x + floor(m/2) + 32 (0 <= u <= m + 64 < 2^12) in 12-bit slots,
// the lane's 16 outputs of a 32x32 block as two 96-bit records (outputs
// 8h .. 8h+7 in record h, output 8h + e at bits 12 e); lane-major here
// (the lane's six words at 6 L: accumulate reads them so), pair-major in
// the short-k kernel (store_residues_pair).  fin is a power of
// two, so the reduction runs on acc itself: RN(acc * (fin RN(1/m))) =
// RN(v * RN(1/m)), the same quotient q; acc - q (m/fin) = x/fin is exact, and
// the fma that adds the offset restores x.  Two neighbouring slots are formed
// as one integer u0 + 4096 u1 < 2^24 by two more fmas (exact) and one
// conversion.  dst: the lane's records of the wave's 128 x 64 outputs.
__device__ __forceinline__ void pack_residues(const Oz2Const& c, int mi, const v16f (&acc)[4][2],
                                              int accumulate, const uint32_t* dst,
                                              uint32_t (&pk)[4][2][6]) {
  const int m = c.m[mi];
  const float fm = (float)m, inv = c.finv[mi];
  const float ffin = (float)c.fin[mi];
  const int offi = m / 2 + 32;
  const float finv = inv * ffin, fmf = fm / ffin;
  // the scale of r16 at packing time: x/fin, or x after the slab sum
  const float pf = accumulate ? 1.0f : ffin;
  const float off1 = (float)offi, off2 = (float)(offi * 4097);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float r16[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float a = acc[i][j][e];
        r16[e] = __builtin_fmaf(-rintf(a * finv), fmf, a);
      }
      if (accumulate) {
        const uint2* p = reinterpret_cast<const uint2*>(dst + (i * 2 + j) * 384);
        const uint2 o0 = p[0], o1 = p[1], o2 = p[2];
        const uint32_t ow[7] = {o0.x, o0.y, o1.x, o1.y, o2.x, o2.y, 0u};
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          // slot e % 8 of record e / 8 (words 3 (e / 8) ..)
          const int bit = 96 * (e >> 3) + 12 * (e & 7), wi = bit >> 5, sh = bit & 31;
          const uint32_t u = (sh + 12 <= 32 ? (ow[wi] >> sh)
                                            : __builtin_amdgcn_alignbit(ow[wi + 1], ow[wi], sh)) &
                             0xFFFu;
          const float t = r16[e] * ffin + (float)((int)u - offi);
          r16[e] = __builtin_fmaf(-rintf(t * inv), fm, t);
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float* x8 = r16 + 8 * h;
        // u_e = x_e + offi; p_ab = u_a + 4096 u_b
        const uint32_t p01 = (uint32_t)__builtin_fmaf(x8[1], pf * 4096.0f,
                                                      __builtin_fmaf(x8[0], pf, off2));
        const uint32_t p34 = (uint32_t)__builtin_fmaf(x8[4], pf * 4096.0f,
                                                      __builtin_fmaf(x8[3], pf, off2));
        const uint32_t p67 = (uint32_t)__builtin_fmaf(x8[7], pf * 4096.0f,
                                                      __builtin_fmaf(x8[6], pf, off2));
        const uint32_t u2 = (uint32_t)__builtin_fmaf(x8[2], pf, off1);
        const uint32_t u5 = (uint32_t)__builtin_fmaf(x8[5], pf, off1);
        pk[i][j][3 * h] = p01 | (u2 << 24);
        pk[i][j][3 * h + 1] = (u2 >> 8) | (p34 << 4) | (u5 << 28);
        pk[i][j][3 * h + 2] = (u5 >> 4) | (p67 << 8);
      }
    }
}

// The non-temporal stores of pack_residues' records: nothing in the launch
// reads them, and with a short k (a few stages per modulus) they drain
// measurably faster.
__device__ __forceinline__ void store_residues(uint32_t* dst, const uint32_t (&pk)[4][2][6]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      u32x2* p = reinterpret_cast<u32x2*>(dst + (i * 2 + j) * 384);
#pragma unroll
      for (int q = 0; q < 3; ++q)
        __builtin_nontemporal_store(u32x2{pk[i][j][2 * q], pk[i][j][2 * q + 1]}, p + q);
    }
}

// The short-k kernel's records, pair-major (oz2_pair_records): word pair q
// of lane L at 8-byte slot 64 q + L of the block, so that each of the three
// non-temporal stores writes 512 consecutive bytes.  wb: the wave's records
// (8 blocks of 384 words).
__device__ __forceinline__ void store_residues_pair(uint32_t* wb, const uint32_t (&pk)[4][2][6]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      u32x2* p = reinterpret_cast<u32x2*>(wb + (i * 2 + j) * 384) + lane;
#pragma unroll
      for (int q = 0; q < 3; ++q)
        __builtin_nontemporal_store(u32x2{pk[i][j][2 * q], pk[i][j][2 * q + 1]}, p + 64 * q);
    }
}

// ------------------------------------------------------------- residue GEMM
// grid: (tiles tbase .. tbase + gridDim.x - 1, 1).  Workgroup t computes
// moduli mgroup*mpw .. min(r, (mgroup+1)*mpw) - 1 of tile tbase + t over k in
// [kbeg, kend), one after the other on one accumulator set, as one
// continuous DMA stream.
// CH bit 0: square moduli, bit 1: nonsquare moduli take the first chain
// transition as a plain multiply (every modulus of that kind has k <= kcheap)
template <int CH>
__global__ void __launch_bounds__(NT, 1)
k_resgemm(Oz2Const c, const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, int mp,
          int np, int kp, int kbeg, int kend, int accumulate, int mpw, int mgroup, int tbase,
          uint32_t* __restrict__ res) {
  __shared__ __attribute__((aligned(16))) uint8_t LB[NB * STB];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u8*)LB;
  const int ntm = mp / TILE, ntn = np / TILE;
  const int tile = tile_of(tbase + blockIdx.x, ntm, ntn);
  const int mi0 = mgroup * mpw, mi1 = min(c.r, mi0 + mpw);
  const int tm = tile % ntm, tn = tile / ntm;
  Ctx x;
  x.psA = (size_t)mp * kp;
  x.psB = (size_t)np * kp;
  x.kbA = (size_t)mp * KS;
  x.kbB = (size_t)np * KS;
  x.a0 = PA + (size_t)tm * TILE * KS + (size_t)(kbeg / KS) * x.kbA;
  x.b0 = PB + (size_t)tn * TILE * KS + (size_t)(kbeg / KS) * x.kbB;
  x.nk = (kend - kbeg) / KS;
  x.T = 3 * x.nk * (mi1 - mi0);
  x.mi1 = mi1;
  const int nk = x.nk;
  Dma dm = dma_init(x);
  dm.mi = mi0;
  product_ptrs(&c, x, mi0, 0, dm);
  const int g = __builtin_amdgcn_readfirstlane(threadIdx.x >> 8);
  prologue<true>(&c, x, dm, lds0, g);

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int it = 0, landed = 0;
  for (int mi = mi0; mi < mi1; ++mi) {
    const int m = c.m[mi], s = c.sq[mi];
    const float fm = (float)m, inv = c.finv[mi];
    v16f acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = v16f{0.f};

    // chain transitions: acc <- (acc - m rint(acc/m)) * rho.  The reduced
    // value has magnitude <= m/2 + 3 (the fp32 quotient estimate is within 1
    // of the exact one), so |acc * rho| < 2^18 and the next pair keeps every
    // partial sum below 2^24.  Square moduli: the two cross products share
    // one chain (their sum is at most 512 k_slab = 2^24), then x s before
    // d0e0.  Nonsquare: d1e1, x rho0 = 240/(-15), d0e0, x rho1 = -15/16,
    // (d0+d1)(e0+e1).
    // short chains (k <= kcheap) need no reduction at the first transition:
    // a plain multiply by the integer coefficient ratio keeps them exact
    if (s) {
      run_stages<true>(&c, x, dm, LB, lds0, it, 2 * nk, landed, g, acc);
      if (CH & 1) chain_scale(acc, (float)s);
      else chain_reduce(acc, inv, fm, (float)s);
      run_stages<true>(&c, x, dm, LB, lds0, it + 2 * nk, nk, landed, g, acc);
    } else {
      run_stages<true>(&c, x, dm, LB, lds0, it, nk, landed, g, acc);
      if (CH & 2) chain_scale(acc, -16.0f);
      else chain_reduce(acc, inv, fm, (float)c.rho0[mi]);
      run_stages<true>(&c, x, dm, LB, lds0, it + nk, nk, landed, g, acc);
      chain_reduce(acc, inv, fm, (float)c.rho1[mi]);
      run_stages<true>(&c, x, dm, LB, lds0, it + 2 * nk, nk, landed, g, acc);
    }
    it += 3 * nk;

    uint32_t* dst = res + ((size_t)mi * mp * np + (size_t)tile * (TILE * TILE) +
                           (size_t)w * 8192) / 8 * 3 + lane * 6;
    uint32_t pk[4][2][6];
    pack_residues(c, mi, acc, accumulate, dst, pk);
    // Every DMA issued so far (the next modulus's first stages, up to three)
    // has landed before the stores go out; those stages then skip their wait,
    // and the wait of the stage after them also covers the stores.
    wait_vm<0>();
    landed = it + 3;
    store_residues(dst, pk);
  }
  if (!g) bar();
  wait_vm<0>();
}


// ------------------------------------------- residue GEMM, two workgroups per CU
// For short k (a workgroup walks many moduli of its tile, each a handful of
// K-stages) the per-modulus work outside the MFMAs -- chain transitions, the
// epilogue and its stores -- is as long as the modulus's MFMAs, and the
// lockstep ping-pong of k_resgemm cannot overlap it.  This variant gives each
// CU two independent workgroups instead: 256 threads (4 waves, 1 per SIMD),
// one 256 x 128 half of a 256 x 256 tile, a 3-deep ring of 24 KiB stages
// (72 KiB of LDS), one barrier per stage.  While one workgroup's waves run a
// transition, an epilogue or wait for LDS, the other's keep the SIMDs'
// matrix units busy.  Wave v computes the same 128 x 64 outputs (and stores
// them in the same blocks, pair-major) as wave w = 4 (v / 2) + 2 h + v % 2 of
// k_resgemm for half h.  The DMA stream: stage = A tile (16 blocks of 16 rows x 64 B)
// + the half's B tile (8 blocks); wave v moves A blocks v + 4j (j < 4) and B
// blocks v + 4j (j < 2).
constexpr int DSTB = OPB + OPB / 2;   // 24 KiB per stage
constexpr int DNB = 3;                // ring depth
constexpr int DNT = 256;

struct DuoDma {
  const uint8_t* pa;
  const uint8_t* pb;
  int left, q, mi;
  uint32_t vo;   // lane offset of block v in a stage (VGPR)
  uint32_t mv;   // v * 1 KiB (uniform)
};

__device__ __forceinline__ void duo_issue(const Oz2Const* c, const Ctx& x, DuoDma& d,
                                          uint32_t lbase) {
#pragma unroll
  for (int j = 0; j < 4; ++j) dma16(d.pa + 4096 * j, d.vo, lbase + d.mv + 4096u * j);
#pragma unroll
  for (int j = 0; j < 2; ++j) dma16(d.pb + 4096 * j, d.vo, lbase + OPB + d.mv + 4096u * j);
  d.pa += x.kbA;
  d.pb += x.kbB;
  if (--d.left == 0) {
    d.left = x.nk;
    if (++d.q == 3) {
      d.q = 0;
      ++d.mi;
    }
    if (d.mi < x.mi1) {
      const int s = c->sq[d.mi], p0 = c->pbase[d.mi];
      d.pa = x.a0 + (size_t)(p0 + planeA(s, d.q)) * x.psA;
      d.pb = x.b0 + (size_t)(p0 + planeB(s, d.q)) * x.psB;
    }
  }
}

// Stages [it0, it0 + n): wait for this wave's share of stage t (issued two
// stages ahead: six DMA instructions per stage, returning in order; stages
// below `landed` are known to be in LDS), barrier (every share of stage t
// landed, every wave done reading stage t - 1), refill the slot of stage
// t - 1 with stage t + 2, then the fragments and the 8 MFMAs of stage t.
__device__ __forceinline__ void duo_run(const Oz2Const* c, const Ctx& x, DuoDma& dm,
                                        const uint8_t* LB, uint32_t lds0, int it0, int n,
                                        int landed, int wr, int wc, v16f (&acc)[4][2]) {
  const int T = x.T;
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, sw = swz(lane & 31);
  const int o0 = 16 * ((2 * h) ^ sw), o1 = 16 * ((2 * h + 1) ^ sw);
  for (int it = it0; it < it0 + n; ++it) {
    if (it >= landed) {
      if (it + 1 < T) wait_vm<6>();
      else wait_vm<0>();
    }
    bar();
    if (it + 2 < T) duo_issue(c, x, dm, lds0 + ((it + 2) % DNB) * DSTB);
    const uint8_t* st = LB + (it % DNB) * DSTB;
    const uint8_t* sa = st + (wr * 128 + (lane & 31)) * KS;
    const uint8_t* sb = st + OPB + (wc * 64 + (lane & 31)) * KS;
    v8i fa[4], fb[2];
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[i] = ldfrag(sa + i * 32 * KS, o0, o1);
#pragma unroll
    for (int j = 0; j < 2; ++j) fb[j] = ldfrag(sb + j * 32 * KS, o0, o1);
    wait_lgkm0();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa[i], fb[j], acc[i][j], 0, 0,
                                                                   0, 0, 0, 0);
  }
}

// grid: 2 x (tiles tbase .. tbase + gridDim.x / 2 - 1), the two halves of a
// tile on the same XCD (blocks b and b + 8); the tile count of a launch is a
// multiple of 8.
template <int CH>
__global__ void __launch_bounds__(DNT, 2)
k_resgemm_duo(Oz2Const c, const uint8_t* __restrict__ PA, const uint8_t* __restrict__ PB, int mp,
              int np, int kp, int kbeg, int kend, int accumulate, int mpw, int mgroup, int tbase,
              uint32_t* __restrict__ res) {
  extern __shared__ __attribute__((aligned(16))) uint8_t LB[];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u8*)LB;
  const int ntm = mp / TILE, ntn = np / TILE;
  const int b = blockIdx.x, slot = b >> 3, half = slot & 1;
  const int tile = tile_of(tbase + (slot >> 1) * 8 + (b & 7), ntm, ntn);
  const int mi0 = mgroup * mpw, mi1 = min(c.r, mi0 + mpw);
  const int tm = tile % ntm, tn = tile / ntm;
  Ctx x;
  x.psA = (size_t)mp * kp;
  x.psB = (size_t)np * kp;
  x.kbA = (size_t)mp * KS;
  x.kbB = (size_t)np * KS;
  x.a0 = PA + (size_t)tm * TILE * KS + (size_t)(kbeg / KS) * x.kbA;
  x.b0 = PB + (size_t)(tn * TILE + half * (TILE / 2)) * KS + (size_t)(kbeg / KS) * x.kbB;
  x.nk = (kend - kbeg) / KS;
  x.T = 3 * x.nk * (mi1 - mi0);
  x.mi1 = mi1;
  const int nk = x.nk;
  const int lane = threadIdx.x & 63;
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = v >> 1, wc = v & 1, w = 4 * wr + 2 * half + wc;
  DuoDma dm;
  {
    const int rb = lane >> 2;
    dm.vo = (uint32_t)(rb * KS + 16 * ((lane & 3) ^ swz(rb))) + (uint32_t)v * 1024u;
    dm.mv = (uint32_t)v * 1024u;
    dm.left = nk;
    dm.q = 0;
    dm.mi = mi0;
    const int s = c.sq[mi0], p0 = c.pbase[mi0];
    dm.pa = x.a0 + (size_t)(p0 + planeA(s, 0)) * x.psA;
    dm.pb = x.b0 + (size_t)(p0 + planeB(s, 0)) * x.psB;
  }
  for (int t = 0; t < DNB - 1; ++t)
    if (t < x.T) duo_issue(&c, x, dm, lds0 + t * DSTB);

  int it = 0, landed = 0;
  for (int mi = mi0; mi < mi1; ++mi) {
    const int m = c.m[mi], s = c.sq[mi];
    const float fm = (float)m, inv = c.finv[mi];
    v16f acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = v16f{0.f};
    // the chains of k_resgemm
    if (s) {
      duo_run(&c, x, dm, LB, lds0, it, 2 * nk, landed, wr, wc, acc);
      if (CH & 1) chain_scale(acc, (float)s);
      else chain_reduce(acc, inv, fm, (float)s);
      duo_run(&c, x, dm, LB, lds0, it + 2 * nk, nk, landed, wr, wc, acc);
    } else {
      duo_run(&c, x, dm, LB, lds0, it, nk, landed, wr, wc, acc);
      if (CH & 2) chain_scale(acc, -16.0f);
      else chain_reduce(acc, inv, fm, (float)c.rho0[mi]);
      duo_run(&c, x, dm, LB, lds0, it + nk, nk, landed, wr, wc, acc);
      chain_reduce(acc, inv, fm, (float)c.rho1[mi]);
      duo_run(&c, x, dm, LB, lds0, it + 2 * nk, nk, landed, wr, wc, acc);
    }
    it += 3 * nk;
    uint32_t* wb = res + ((size_t)mi * mp * np + (size_t)tile * (TILE * TILE) +
                          (size_t)w * 8192) / 8 * 3;
    uint32_t pk[4][2][6];
    pack_residues(c, mi, acc, 0, wb, pk);   // a single slab: nothing to add
    // the DMAs issued so far (the next modulus's first two stages) land
    // before the stores go out; those stages skip their wait, and the wait
    // of the stage after them also covers the stores
    wait_vm<0>();
    landed = it + 2;
    store_residues_pair(wb, pk);
  }
  wait_vm<0>();
}

}  // namespace

// Launch granularity: one modulus group and a few rounds of tiles per
// launch.  The workgroups of an XCD that share A or B panels (the 4 x 8
// groups of tile_of) run their K-loops in step only while they started
// together: in one long launch the dispatcher refills each CU as its
// workgroup ends, their starts drift apart round after round, and the shared
// panel blocks no longer meet in L2.  A new launch starts them together
// again (16384^3 at r = 15: 56.2 -> 61.8 TF on one box with four rounds per
// launch; one launch per modulus alone gave 61.3).  Each launch also costs a
// ramp-up and a tail, so a launch holds one round when a workgroup's run is
// long (+0.5% at 16384^3) and four when it is short (one round per launch
// lost 4.6% on 32768^2 x 256).  Chunks are whole multiples of 256 tiles, so
// that tbase keeps the XCD of every workgroup and the 4 x 8 groups whole.
static int launch_tiles(int rounds) {
  return std::max(256, (rounds * oz2_device_cus() + 255) / 256 * 256);
}

hipError_t oz2_launch_codegemm(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, hipStream_t s) {
  const int tiles = (d.mp / TILE) * (d.np / TILE);
  const int chunk = launch_tiles(4);
  for (int tb = 0; tb < tiles; tb += chunk) {
    dim3 grid(std::min(chunk, tiles - tb), d.cslabs);
    hipLaunchKernelGGL(k_codegemm, grid, dim3(NT), 0, s, ws + L.codesA, ws + L.codesB, d.mp,
                       d.np, d.kp, (uint32_t*)(ws + L.Rmax), (uint32_t*)(ws + L.Kmax), tb);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t oz2_launch_resgemm(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                              uint8_t* ws, hipStream_t s) {
  // moduli per workgroup.  Enough groups that tiles x groups covers the
  // device (one resident workgroup per CU), and no more than about WG_STEPS
  // K-steps of plane products (three per modulus) in one workgroup: the CUs
  // run at slightly different clocks, and the dispatcher evens that out only
  // when a workgroup is a small share of a CU's work.  A short k keeps all
  // moduli together, since each workgroup pays a prologue and an epilogue.
  constexpr int WG_STEPS = 768;
  const int cus = oz2_device_cus();
  const int tiles = (d.mp / TILE) * (d.np / TILE);
  const int fill = std::min(c.r, (cus + tiles - 1) / tiles);
  const int ksteps = (std::min(d.kp, OZ2_KSLAB) + KS - 1) / KS;
  const int by_work = std::max(1, WG_STEPS / (3 * ksteps));
  const int mpw = std::min((c.r + fill - 1) / fill, by_work);
  const int groups = (c.r + mpw - 1) / mpw;
  const int chunk = launch_tiles(3 * ksteps * mpw >= WG_STEPS / 2 ? 1 : 4);
  for (int kb = 0, sl = 0; kb < d.kp; kb += OZ2_KSLAB, ++sl) {
    const int ke = kb + OZ2_KSLAB < d.kp ? kb + OZ2_KSLAB : d.kp;
    // the first chain transition may skip its reduction when every modulus of
    // a kind has k <= kcheap for this slab
    bool sq_cheap = true, ns_cheap = true;
    for (int i = 0; i < c.r; ++i) {
      const bool ok = ke - kb <= c.kcheap[i];
      if (c.sq[i]) sq_cheap = sq_cheap && ok;
      else ns_cheap = ns_cheap && ok;
    }
    const int ch = (sq_cheap ? 1 : 0) | (ns_cheap ? 2 : 0);
    typedef void (*Kern)(Oz2Const, const uint8_t*, const uint8_t*, int, int, int, int, int, int,
                         int, int, int, uint32_t*);
    const bool duo = oz2_pair_records(d);
    Kern kern = duo ? (ch == 3 ? k_resgemm_duo<3> : ch == 2 ? k_resgemm_duo<2>
                       : ch == 1 ? k_resgemm_duo<1> : k_resgemm_duo<0>)
                    : (ch == 3 ? k_resgemm<3> : ch == 2 ? k_resgemm<2>
                       : ch == 1 ? k_resgemm<1> : k_resgemm<0>);
    const int lds = duo ? DNB * DSTB : 0;
    if (duo) (void)hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    for (int g = 0; g < groups; ++g)
      for (int tb = 0; tb < tiles; tb += chunk) {
        const int nt = std::min(chunk, tiles - tb);
        hipLaunchKernelGGL(kern, dim3(duo ? 2 * nt : nt), dim3(duo ? DNT : NT), lds, s, c,
                           ws + L.planesA, ws + L.planesB, d.mp, d.np, d.kp, kb, ke,
                           sl > 0 ? 1 : 0, mpw, g, tb, (uint32_t*)(ws + L.res));
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
      }
  }
  return hipSuccess;
}
