// Phase 3 of Alg. 1 on gfx950: CRT reconstruction of the exact integer,
// removal of the power-of-two scaling with ONE rounding of the multi-limb
// integer (App. B), and the native-FP64 fallback for flagged rows of A /
// columns of B (Alg. 1, fallback step: rows the scaling cannot certify are
// recomputed in plain FP64; the numerical contract's item (vi)).
//
// Reconstruction.  The integer C~ in [-M/2, M/2) is unique given its r
// residues (Eq. (M-bound)), so any exact CRT algorithm yields the same bits
// as Garner's Eq. (garner).  On this VALU the direct CRT sum is cheaper than
// Garner's r(r-1)/2 dependent modular steps:
//     X = sum_i x_i W_i - q M,  W_i = (M/m_i) ((M/m_i)^-1 mod m_i),
// evaluated exactly in radix-2^38 fp64 limbs (three for r <= 12, four
// above), with q = rint(sum_i x_i W_i/M) estimated from the top limbs (error
// < 2^-24; an exact range check fixes the rare ambiguous case).  The x_i are
// any representatives of the residues with |x_i| <= m_i/2 + 32 <= 577 (what
// the residue GEMM stores): every partial limb sum is then an integer below
// 2^52, and the quotient estimate is as good for them as for centred
// residues.  The residue GEMMs store them offset (u = x + floor(m/2) + 32,
// 12 bits per output): the sums start at minus the offsets' share and add the
// u_i, which gives the same integers.
// The normalised limbs are rounded once to binary64 with the exponent shift
// -(s_i + t_j), including gradual underflow (through 32-bit words) and
// overflow.
#include "oz2_device.h"

namespace {

// Thread mapping shared by the reconstruction kernels.  The residue GEMM
// leaves, per modulus, each 32x32 output block (wave w of a 256x256 tile,
// sub-block x, y) as 1024 12-bit slots in its accumulator order: lane L holds
// 16 outputs of column L%32, rows 4(L/32) + 8(e/4) + e%4, e = 0..15, as two
// 96-bit records (e = 0..7, e = 8..15), six words w = 0..5 per lane, stored
// lane-major or pair-major (oz2_pair_records).  Here two threads share a
// lane's 16 (t = 2L + h takes record h: words 3h .. 3h + 2), so the 128
// threads of a block read its 1.5 KiB per modulus; a workgroup of 256 takes
// two blocks.
struct BlockMap {
  size_t roff;      // word offset of the block in a modulus plane
  int lane, h;      // the record: lane L's record h
  int row0, col0;   // block origin in C
  int cl;           // column within the block
  int rb;           // row within the block of output i: rb + 8(i/4) + i%4
  int hb, tt;       // block of the pair, thread within the block
};

__device__ __forceinline__ BlockMap block_map(int mp) {
  BlockMap b;
  const int t = threadIdx.x;
  b.hb = t >> 7;
  b.tt = t & 127;
  const size_t G = (size_t)blockIdx.x * 2 + b.hb;
  const size_t tile = G >> 6;
  const int blk = (int)(G & 63);
  const int ntm = mp / OZ2_TILE;
  const int tm = (int)(tile % ntm), tn = (int)(tile / ntm);
  const int y = blk & 1, x = (blk >> 1) & 3, w = blk >> 3;
  b.row0 = tm * OZ2_TILE + (w >> 2) * 128 + x * 32;
  b.col0 = tn * OZ2_TILE + (w & 3) * 64 + y * 32;
  const int lane = b.tt >> 1, h = b.tt & 1;
  b.cl = lane & 31;
  b.rb = 4 * (lane >> 5) + 16 * h;
  b.roff = tile * (OZ2_TILE * OZ2_TILE / 8 * 3) + (size_t)blk * 384;
  b.lane = lane;
  b.h = h;
  return b;
}

// the thread's record of each modulus (plane: words per modulus).
// Lane-major: words 6 L + 3 h .. + 2, one 12-byte load.  Pair-major: record
// 0 is words 0, 1 (8 bytes at 2 L) and 2 (at 128 + 2 L), record 1 words 3
// (at 129 + 2 L) and 4, 5 (8 bytes at 256 + 2 L).  The residues, C_in and C
// are each touched once: non-temporal loads and stores (3-4% faster
// reconstruction on the 16384^3 and rank-256 workloads).
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
template <int R, bool PAIR>
__device__ __forceinline__ void load_residues(const uint32_t* __restrict__ res, size_t plane,
                                              const BlockMap& b, uint3 (&x)[R]) {
  if constexpr (PAIR) {
    const int o2 = b.h ? 256 + 2 * b.lane : 2 * b.lane, o1 = 128 + 2 * b.lane + b.h;
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const uint32_t* q = res + (size_t)i * plane + b.roff;
      const u32x2 p = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(q + o2));
      const uint32_t w = __builtin_nontemporal_load(q + o1);
      x[i] = b.h ? make_uint3(w, p.x, p.y) : make_uint3(p.x, p.y, w);
    }
  } else {
    const int o = 6 * b.lane + 3 * b.h;
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const uint32_t* q = res + (size_t)i * plane + b.roff + o;
      x[i] = make_uint3(__builtin_nontemporal_load(q), __builtin_nontemporal_load(q + 1),
                        __builtin_nontemporal_load(q + 2));
    }
  }
}

template <int R, int I>
struct Outputs {
  __device__ __forceinline__ static void run(const Oz2Const& c, const Oz2Dims& d,
                                             const uint3 (&x)[R], const BlockMap& b, int tj,
                                             const int32_t* __restrict__ sA, double (*tr)[33]) {
    const int rr = b.rb + 8 * (I >> 2) + (I & 3);
    const int row = b.row0 + rr;
    const int si = row < d.m ? sA[row] : 0;
    tr[b.cl][rr] = crt38_rounded<R, I>(c, x, si + tj);
    Outputs<R, I + 1>::run(c, d, x, b, tj, sA, tr);
  }
};
template <int R>
struct Outputs<R, 8> {
  __device__ __forceinline__ static void run(const Oz2Const&, const Oz2Dims&, const uint3 (&)[R],
                                             const BlockMap&, int, const int32_t* __restrict__,
                                             double (*)[33]) {}
};

// Reconstruct, rescale and store: the block's 32x32 results go through LDS so
// that each store instruction writes whole 256-byte column segments of C.
// Entries of flagged rows / columns are left to the fallback kernel, which
// follows on the same stream; for it the grid also gathers the first `cap`
// flagged rows of A into a contiguous panel (row r at panel[r + l cap]), read
// once here instead of once per column tile there (nothing to do on inputs
// without flagged rows).  ACC (OZ2_ACCUMULATE): C_in is loaded before the
// CRT work, so that its latency hides behind it.  PAIR: the records are
// pair-major (oz2_pair_records; a separate instantiation, which measured
// 0.4 ms faster on the rank-256 update than one kernel reading both).
template <int R, bool ACC, bool PAIR>
__global__ void __launch_bounds__(256)
k_reconstruct(Oz2Const c, Oz2Dims d, const uint32_t* __restrict__ res,
              const int32_t* __restrict__ sA, const int32_t* __restrict__ tB,
              const uint32_t* __restrict__ fA, const uint32_t* __restrict__ fB, double* C, int ldc,
              const double* __restrict__ A, int lda, const int* __restrict__ counters,
              const int* __restrict__ listA, double* __restrict__ panel, int cap) {
  __shared__ double tr[2][32][33];
  const int nflag = panel ? counters[0] : 0;   // used at the end; loaded early
  const BlockMap b = block_map(d.mp);
  const int rr = b.tt & 31;
  const int row = b.row0 + rr;
  // the thread's outputs in the store phase: row, columns col0 + 4 j + tt/32
  double cin[8];
  if constexpr (ACC) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int col = b.col0 + j * 4 + (b.tt >> 5);
      cin[j] = (row < d.m && col < d.n) ? __builtin_nontemporal_load(C + (size_t)col * ldc + row) : 0.0;
    }
  }
  {
    uint3 x[R];
    load_residues<R, PAIR>(res, (size_t)d.mp * d.np / 8 * 3, b, x);
    const int col = b.col0 + b.cl;
    const int tj = col < d.n ? tB[col] : 0;
    Outputs<R, 0>::run(c, d, x, b, tj, sA, tr[b.hb]);
  }
  __syncthreads();
  const bool nofb = (d.flags & 8u) != 0;       // OZ2_NO_FALLBACK
  const bool force = (d.flags & 16u) != 0;     // OZ2_FORCE_FALLBACK
  if (row < d.m && !(!nofb && (force || (fA[row] & (OZ2_T1 | OZ2_T2))))) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int cc = j * 4 + (b.tt >> 5);
      const int col = b.col0 + cc;
      if (col < d.n && (nofb || !(fB[col] & (OZ2_T1 | OZ2_T2)))) {
        const double v = tr[b.hb][cc][rr];
        __builtin_nontemporal_store(ACC ? cin[j] + v : v, C + (size_t)col * ldc + row);
      }
    }
  }
  // the fallback's panel: grid-stride over (row of the list, k)
  const int na = min(nflag, cap);
  const size_t total = (size_t)na * d.k, step = (size_t)gridDim.x * blockDim.x;
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += step) {
    const size_t l = idx / na;
    const int r = (int)(idx - l * na);
    panel[r + l * cap] = A[(size_t)listA[r] + l * lda];
  }
}

// The exact integer of output I of a thread as NL 32-bit words (two's
// complement, little endian), formed by the routine the reconstruction
// itself uses: radix-2^38 limbs (three for R <= 12, four above).
template <int R, int I, class X>
__device__ __forceinline__ void store_integer(const Oz2Const& c, const X (&x)[R], uint32_t* o) {
  constexpr int NB = Limbs38<R>::value, NW = NB + 1;
  static_assert(NW <= NL, "the exported words hold the limbs");
  uint32_t w[NW];
  double S[NB];
  crt38_limbs<R, I, NB>(c, x, S);
  limbs38_words<NB>(S, w);
  const uint32_t ext = (uint32_t)((int32_t)w[NW - 1] >> 31);
#pragma unroll
  for (int q = 0; q < NL; ++q) o[q] = q < NW ? w[q < NW ? q : 0] : ext;
}

// The rounded value of output I exactly as the reconstruction forms it.
template <int R, int I, class X>
__device__ __forceinline__ double rounded_value(const Oz2Const& c, const X (&x)[R], int e) {
  return crt38_rounded<R, I>(c, x, e);
}

template <int R, int I>
struct IntOut {
  __device__ __forceinline__ static void run(const Oz2Const& c, const Oz2Dims& d,
                                             const uint3 (&x)[R], const BlockMap& b,
                                             uint32_t* out) {
    const int row = b.row0 + b.rb + 8 * (I >> 2) + (I & 3);
    const int col = b.col0 + b.cl;
    if (row < d.m && col < d.n) {
      uint32_t* o = out + ((size_t)col * d.m + row) * NL;
      store_integer<R, I>(c, x, o);
    }
    IntOut<R, I + 1>::run(c, d, x, b, out);
  }
};
template <int R>
struct IntOut<R, 8> {
  __device__ __forceinline__ static void run(const Oz2Const&, const Oz2Dims&, const uint3 (&)[R],
                                             const BlockMap&, uint32_t*) {}
};

// the exact integers themselves, [n][m][5] words (a diagnostic query)
template <int R>
__global__ void __launch_bounds__(256)
k_integers(Oz2Const c, Oz2Dims d, const uint32_t* __restrict__ res, uint32_t* out) {
  const BlockMap b = block_map(d.mp);
  uint3 x[R];
  if (oz2_pair_records(d)) load_residues<R, true>(res, (size_t)d.mp * d.np / 8 * 3, b, x);
  else load_residues<R, false>(res, (size_t)d.mp * d.np / 8 * 3, b, x);
  IntOut<R, 0>::run(c, d, x, b, out);
}

// The reconstruction's integer and rounding routines on given residues (a
// probe): thread t takes residue t of each modulus (res[i n + t], any
// representative x with -(floor(m/2) + 32) <= x <= m/2 + 32, what the residue
// GEMMs store), puts it into a stored record as the residue GEMMs do, and
// writes the exact integer as 5 words and its value rounded with the shift e[t].
template <int R>
__global__ void __launch_bounds__(256)
k_crt_probe(Oz2Const c, const int16_t* __restrict__ res, const int* __restrict__ e, int n,
            uint32_t* __restrict__ words, double* __restrict__ rounded) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n) return;
  uint3 x[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int u = (int)res[(size_t)i * n + t] + c.m[i] / 2 + 32;   // slot 0 of the record
    x[i] = make_uint3((uint32_t)u & 0xFFFu, 0u, 0u);
  }
  store_integer<R, 0>(c, x, words + (size_t)t * NL);
  rounded[t] = rounded_value<R, 0>(c, x, e[t]);
}

// Native FP64 for flagged entries.  Work = (flagged rows of A) x (all
// columns) + (all unflagged rows) x (flagged columns of B), in 64 x 64 output
// tiles walked by a grid-stride loop over the device-side counts (no host
// synchronisation; every workgroup exits when the tiles are exhausted).  A
// tile stages 64 rows x 32 k of A and 32 k x 64 columns of B through LDS (the
// next slab's loads held in registers while the current one is multiplied);
// each wave owns a 32 x 32 quarter as 2 x 2 blocks of
// v_mfma_f64_16x16x4_f64: A[i][k] from lane i + 16 k, B[k][j] from lane
// j + 16 k, and D[i][j] in lane j + 16 (i % 4), element i / 4.  The products
// and sums are FP64 in a fixed order (deterministic, not the order of a
// sequential dot product): the result lies within the FP64 dot-product
// error bound, which is the contract for flagged entries.
constexpr int FB_T = 64, FB_K = 32;
typedef double v4d __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256)
k_fallback(Oz2Dims d, const double* __restrict__ A, int lda, const double* __restrict__ B, int ldb,
           double* C, int ldc, const int* __restrict__ counters, const int* __restrict__ listA,
           const int* __restrict__ listB, const uint32_t* __restrict__ fA,
           const double* __restrict__ panel, int cap) {
  __shared__ double sa[FB_K][FB_T + 2];   // [k][row]
  __shared__ double sb[FB_K][FB_T + 2];   // [k][column]
  __shared__ int rowid[FB_T], colid[FB_T], arow[FB_T];
  const int na = counters[0], nb = counters[1];
  const bool acc = (d.flags & 1u) != 0;
  const bool force = (d.flags & 16u) != 0;
  // part 1: ceil(na/64) x ceil(n/64) tiles; part 2: ceil(m/64) x ceil(nb/64) tiles
  const int t1r = (na + FB_T - 1) / FB_T, t1c = (d.n + FB_T - 1) / FB_T;
  const int t2r = (d.m + FB_T - 1) / FB_T, t2c = (nb + FB_T - 1) / FB_T;
  const long long tiles1 = (long long)t1r * t1c, total = tiles1 + (long long)t2r * t2c;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wr = 32 * (w >> 1), wc = 32 * (w & 1);
  const int kr = lane >> 4, cl = lane & 15;
  for (long long tile = blockIdx.x; tile < total; tile += gridDim.x) {
    // A rows come from the gathered panel when the tile's list rows all lie
    // in it (row r of the list at panel[r + l cap]), else from A itself
    const double* As = A;
    int ldas = lda;
    if (tile < tiles1) {
      const int tr = (int)(tile / t1c), tc = (int)(tile % t1c);
      const int nr = min(FB_T, na - tr * FB_T), nc = min(FB_T, d.n - tc * FB_T);
      const bool inpanel = panel != nullptr && (tr + 1) * FB_T <= cap;
      if (inpanel) {
        As = panel;
        ldas = cap;
      }
      if (t < FB_T) {
        rowid[t] = t < nr ? listA[tr * FB_T + t] : -1;
        arow[t] = t < nr ? (inpanel ? tr * FB_T + t : rowid[t]) : -1;
        colid[t] = t < nc ? tc * FB_T + t : -1;
      }
    } else {
      const long long u = tile - tiles1;
      const int tr = (int)(u / t2c), tc = (int)(u % t2c);
      const int nr = min(FB_T, d.m - tr * FB_T), nc = min(FB_T, nb - tc * FB_T);
      if (t < FB_T) {
        const int i = tr * FB_T + t;
        // rows already recomputed in part 1 (flagged rows) are skipped here
        rowid[t] = (t < nr && !(force || (fA[i] & (OZ2_T1 | OZ2_T2)))) ? i : -1;
        arow[t] = rowid[t];
        colid[t] = t < nc ? listB[tc * FB_T + t] : -1;
      }
    }
    __syncthreads();
    // slab loads: thread t takes A entries (row e % 64, k e / 64) and B
    // entries (column e / 32, k e % 32) for e = t + 256 q; outside -> 0
    double pa[8], pb[8];
    auto load = [&](int l0) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int e = t + 256 * q;
        const int i = arow[e & 63], l = l0 + (e >> 6);
        pa[q] = (i >= 0 && l < d.k) ? As[(size_t)i + (size_t)l * ldas] : 0.0;
        const int j = colid[e >> 5], lb = l0 + (e & 31);
        pb[q] = (j >= 0 && lb < d.k) ? B[(size_t)lb + (size_t)j * ldb] : 0.0;
      }
    };
    v4d cacc[2][2];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) cacc[bi][bj] = v4d{0.0, 0.0, 0.0, 0.0};
    load(0);
    for (int l0 = 0; l0 < d.k; l0 += FB_K) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int e = t + 256 * q;
        sa[e >> 6][e & 63] = pa[q];
        sb[e & 31][e >> 5] = pb[q];
      }
      __syncthreads();
      if (l0 + FB_K < d.k) load(l0 + FB_K);
#pragma unroll
      for (int kk = 0; kk < FB_K; kk += 4) {
        const double a0 = sa[kk + kr][wr + cl], a1 = sa[kk + kr][wr + 16 + cl];
        const double b0 = sb[kk + kr][wc + cl], b1 = sb[kk + kr][wc + 16 + cl];
        cacc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, cacc[0][0], 0, 0, 0);
        cacc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, cacc[0][1], 0, 0, 0);
        cacc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, cacc[1][0], 0, 0, 0);
        cacc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, cacc[1][1], 0, 0, 0);
      }
      __syncthreads();
    }
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int i = rowid[wr + 16 * bi + 4 * v + kr], j = colid[wc + 16 * bj + cl];
          if (i >= 0 && j >= 0) {
            double* o = C + (size_t)i + (size_t)j * ldc;
            *o = acc ? *o + cacc[bi][bj][v] : cacc[bi][bj][v];
          }
        }
    __syncthreads();   // rowid / colid are rewritten by the next tile
  }
}

__global__ void k_fill(double* C, int m, int n, int ldc) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)m * n) return;
  const size_t j = idx / m, i = idx % m;
  C[i + j * ldc] = 0.0;
}

// one workgroup of 256 threads per two 32x32 output blocks
template <int R>
void launch_reconstruct_r(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                          const double* A, int lda, double* C, int ldc, hipStream_t s) {
  const size_t blocks = (size_t)d.mp * d.np / 2048;
  const bool gather = !(d.flags & 8u);   // OZ2_NO_FALLBACK: no fallback, no panel
  const bool pair = oz2_pair_records(d);
  auto kern = (d.flags & 1u) ? (pair ? k_reconstruct<R, true, true> : k_reconstruct<R, true, false>)
                             : (pair ? k_reconstruct<R, false, true> : k_reconstruct<R, false, false>);
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, s, c, d,
                     (const uint32_t*)(ws + L.res), (const int32_t*)(ws + L.sA),
                     (const int32_t*)(ws + L.tB), (const uint32_t*)(ws + L.flagsA),
                     (const uint32_t*)(ws + L.flagsB), C, ldc, A, lda,
                     (const int*)(ws + L.counters), (const int*)(ws + L.listA),
                     gather ? (double*)(ws + L.panel) : nullptr, std::min(d.mp, OZ2_FBCAP));
}

template <int R>
void launch_integers_r(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c, uint8_t* ws,
                       uint32_t* out, hipStream_t s) {
  const size_t blocks = (size_t)d.mp * d.np / 2048;
  hipLaunchKernelGGL(k_integers<R>, dim3((unsigned)blocks), dim3(256), 0, s, c, d,
                     (const uint32_t*)(ws + L.res), out);
}

template <int R>
void launch_crt_probe_r(const Oz2Const& c, const int16_t* res, const int* e, int n,
                        uint32_t* words, double* rounded, hipStream_t s) {
  hipLaunchKernelGGL(k_crt_probe<R>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, c, res, e,
                     n, words, rounded);
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
                                  uint8_t* ws, const double* A, int lda, double* C, int ldc,
                                  hipStream_t s) {
  OZ2_R_SWITCH(launch_reconstruct_r, d, L, c, ws, A, lda, C, ldc, s)
  return hipGetLastError();
}

hipError_t oz2_launch_integers(const Oz2Dims& d, const Oz2Layout& L, const Oz2Const& c,
                               uint8_t* ws, uint32_t* out, hipStream_t s) {
  OZ2_R_SWITCH(launch_integers_r, d, L, c, ws, out, s)
  return hipGetLastError();
}


hipError_t oz2_launch_crt_probe(const Oz2Const& c, const int16_t* res, const int* e, int n,
                                uint32_t* words, double* rounded, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  OZ2_R_SWITCH(launch_crt_probe_r, c, res, e, n, words, rounded, s)
  return hipGetLastError();
}

hipError_t oz2_launch_fallback(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws, const double* A,
                               int lda, const double* B, int ldb, double* C, int ldc,
                               hipStream_t s) {
  // the lists were filled by the deconstruction (k_scales: T1, k_split: T2)
  // the panel of flagged rows was gathered by the reconstruction launch
  hipLaunchKernelGGL(k_fallback, dim3(1024), dim3(256), 0, s, d, A, lda, B, ldb, C, ldc,
                     (const int*)(ws + L.counters), (const int*)(ws + L.listA),
                     (const int*)(ws + L.listB), (const uint32_t*)(ws + L.flagsA),
                     (const double*)(ws + L.panel), std::min(d.mp, OZ2_FBCAP));
  return hipGetLastError();
}

hipError_t oz2_launch_fallback_direct(const Oz2Dims& d, const Oz2Layout& L, uint8_t* ws,
                                      const double* A, int lda, const double* B, int ldb,
                                      double* C, int ldc, hipStream_t s) {
  hipLaunchKernelGGL(k_fallback, dim3(1024), dim3(256), 0, s, d, A, lda, B, ldb, C, ldc,
                     (const int*)(ws + L.counters), (const int*)(ws + L.listA),
                     (const int*)(ws + L.listB), (const uint32_t*)(ws + L.flagsA),
                     (const double*)nullptr, 0);
  return hipGetLastError();
}

hipError_t oz2_launch_fill(double* C, int m, int n, int ldc, hipStream_t s) {
  const size_t total = (size_t)m * n;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, C, m, n, ldc);
  return hipGetLastError();
}
