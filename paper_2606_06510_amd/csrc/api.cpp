// Host orchestration of the Ozaki-II FP8 emulated DGEMM (the C ABI of
// include/ozaki2.h): argument validation, the per-plan constant table,
// workspace layout, stage sequencing and test queries.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/ozaki2.h"
#include "../../include/ozaki2_probes.h"
#include "oz2_internal.h"

namespace {

// The paper's r = 12 set S (section "The frozen plane kernel") plus the
// nonsquare extension 481, 479, 467, 463, in descending order; r moduli are
// the r largest, used in ascending order.
const int kPool[OZ2_MAXR] = {1089, 1024, 961, 841, 625, 529, 511, 509,
                             503,  499,  491, 487, 481, 479, 467, 463};

// ------------------------------------------------------------ tiny bigint
struct Big {
  std::vector<uint32_t> w;  // little endian, non-negative
  explicit Big(uint64_t v = 0) {
    w.push_back((uint32_t)v);
    w.push_back((uint32_t)(v >> 32));
    trim();
  }
  void trim() {
    while (w.size() > 1 && w.back() == 0) w.pop_back();
  }
  void mul_small(uint32_t f) {
    uint64_t carry = 0;
    for (auto& x : w) {
      uint64_t t = (uint64_t)x * f + carry;
      x = (uint32_t)t;
      carry = t >> 32;
    }
    if (carry) w.push_back((uint32_t)carry);
    trim();
  }
  uint32_t mod_small(uint32_t m) const {
    uint64_t r = 0;
    for (size_t i = w.size(); i-- > 0;) r = ((r << 32) | w[i]) % m;
    return (uint32_t)r;
  }
  void shr1() {
    for (size_t i = 0; i < w.size(); ++i) {
      w[i] >>= 1;
      if (i + 1 < w.size()) w[i] |= (w[i + 1] & 1u) << 31;
    }
    trim();
  }
  int bitlen() const {
    int top = (int)w.size() - 1;
    while (top > 0 && w[top] == 0) --top;
    if (w[top] == 0) return 0;
    return 32 * top + (32 - __builtin_clz(w[top]));
  }
  uint32_t word(int i) const { return i < (int)w.size() ? w[i] : 0u; }
  // bits lo .. lo+cnt-1 (cnt <= 52) as an integer
  uint64_t bits(int lo, int cnt) const {
    uint64_t v = 0;
    for (int b = cnt - 1; b >= 0; --b) {
      const int pos = lo + b;
      v = (v << 1) | ((word(pos >> 5) >> (pos & 31)) & 1u);
    }
    return v;
  }
};

int64_t inv_mod(int64_t a, int64_t m) {  // a^-1 mod m, gcd(a, m) = 1
  int64_t t = 0, nt = 1, r = m, nr = ((a % m) + m) % m;
  while (nr) {
    int64_t q = r / nr;
    int64_t x = t - q * nt; t = nt; nt = x;
    x = r - q * nr; r = nr; nr = x;
  }
  return t < 0 ? t + m : t;
}

bool build_const(int r, Oz2Const& c) {
  if (r < 8 || r > OZ2_MAXR) return false;
  std::memset(&c, 0, sizeof(c));
  std::vector<int> ms(kPool, kPool + r);
  std::sort(ms.begin(), ms.end());
  c.r = r;
  int pb = 0;
  Big M(1);
  for (int i = 0; i < r; ++i) M.mul_small((uint32_t)ms[i]);
  for (int i = 0; i < r; ++i) {
    const int m = ms[i];
    int s = (int)std::lround(std::sqrt((double)m));
    if (s * s != m) s = 0;
    c.m[i] = m;
    c.sq[i] = s;
    c.pbase[i] = pb;
    pb += s ? 2 : 3;
    c.c32[i] = (int)((1ull << 32) % (uint64_t)m);
    if (s) {
      c.rho0[i] = s;            // chain (d1e0 + d0e1) carries coefficient s, then d0e0 carries 1
      c.rho1[i] = 0;
      c.fin[i] = 1;
    } else {                    // coefficients 240 (d1e1), -15 (d0e0), 16 (sum planes)
      c.rho0[i] = m - 16;                                         // 240 / -15 = -16
      c.rho1[i] = (int)(((int64_t)(m - 15) * inv_mod(16, m)) % m);  // -15 / 16
      c.fin[i] = 16;
    }
    c.finv[i] = 1.0f / (float)m;
    c.finv_s[i] = s ? 1.0f / (float)s : 0.0f;
    c.dinv[i] = 1.0 / (double)m;
    // W_i = (M/m_i) * ((M/m_i)^-1 mod m_i)
    Big Mi(1);
    for (int j = 0; j < r; ++j)
      if (j != i) Mi.mul_small((uint32_t)ms[j]);
    const int64_t inv = inv_mod(Mi.mod_small((uint32_t)m), m);
    Big Wi = Mi;
    Wi.mul_small((uint32_t)inv);
    for (int j = 0; j < OZ2_NLIMB; ++j) c.W[i][j] = (double)Wi.word(j);
    for (int j = 0; j < 4; ++j) c.W38[i][j] = (double)Wi.bits(38 * j, 38);
    Big Wf = Mi;
    Wf.mul_small((uint32_t)((inv * c.fin[i]) % m));
    for (int j = 0; j < 4; ++j) c.W38f[i][j] = (double)Wf.bits(38 * j, 38);
    c.wfrac[i] = (double)inv / (double)m;   // W_i / M exactly = inv_i / m_i
  }
  c.P = pb;
  // kcheap: with digit maxima D0, D1 of the planes (both operands share the
  // digit rule), a k-term chain has |d1 e0 + d0 e1| <= 2 D0 D1 per term and
  // |d0 e0| <= D0^2 (square m: x s between them), or |d1 e1| <= D1^2 and
  // |d0 e0| <= D0^2 (nonsquare m: x -16 between them); an integer multiply
  // keeps the chain exact while k times the bound stays <= 2^24
  for (int i = 0; i < r; ++i) {
    const int m = c.m[i], sq = c.sq[i];
    int D0 = 0, D1 = 0;
    for (int d = -(m / 2); d <= (m + 1) / 2 - 1; ++d) {
      int d0, d1;
      oz2_digits(d, m, sq, d0, d1);
      D0 = std::max(D0, std::abs(d0));
      D1 = std::max(D1, std::abs(d1));
    }
    const long long per = sq ? 2LL * D0 * D1 * sq + (long long)D0 * D0
                             : 16LL * D1 * D1 + (long long)D0 * D0;
    c.kcheap[i] = (int)((1LL << 24) / per);
  }
  int off = 0;
  for (int i = 0; i < r; ++i) {
    c.toff[i] = off + ms[i] / 2;
    off += ms[i];
  }
  c.tabsz = off;
  Big Mh = M;
  Mh.shr1();
  for (int j = 0; j < OZ2_NLIMB; ++j) {
    c.Ml[j] = (double)M.word(j);
    c.Mhalf[j] = (double)Mh.word(j);
  }
  for (int j = 0; j < 4; ++j) {
    c.M38[j] = (double)M.bits(38 * j, 38);
    c.Mhalf38[j] = (double)Mh.bits(38 * j, 38);
  }
  // the reconstruction kernels are specialised on r with nw = 3 (r <= 10),
  // 4 (r <= 13), 5 words: [-M/2, M/2) must fit nw words of two's complement
  c.nw = r <= 10 ? 3 : (r <= 13 ? 4 : 5);
  if (M.bitlen() + 1 > 32 * c.nw) return false;
  double Md = 0.0;
  for (int j = OZ2_NLIMB - 1; j >= 0; --j) Md = Md * 4294967296.0 + (double)M.word(j);
  c.mtop = std::ldexp(1.0, 32 * (c.nw - 1)) / Md;
  // radix-2^38 limbs (the reconstruction): [-M/2, M/2) must fit three limbs
  // (114 bits) for r <= 12 and four (152 bits) above
  const int nl38 = r <= 12 ? 3 : 4;
  if (M.bitlen() + 1 > 38 * nl38) return false;
  c.mtop38 = std::ldexp(1.0, 38 * (nl38 - 1)) / Md;
  // the offsets of the stored residues, folded into the CRT sums
  // (integer sums: W38 limbs < 2^38 and W words < 2^32, offsets <= 576)
  for (int j = 0; j < 4; ++j) {
    int64_t k = 0;
    for (int i = 0; i < r; ++i) k += (int64_t)(ms[i] / 2 + 32) * (int64_t)c.W38[i][j];
    c.K38[j] = (double)k;   // < 2^52: exact
  }
  for (int j = 0; j < OZ2_NLIMB; ++j) {
    int64_t k = 0;
    for (int i = 0; i < r; ++i) k += (int64_t)(ms[i] / 2 + 32) * (int64_t)c.W[i][j];
    c.Kw[j] = (double)k;    // < 2^46: exact
  }
  const int cc = (M.bitlen() - 1) + 6;     // floor(log2 M) + 6
  c.cA = cc / 2;
  c.cB = cc - c.cA;
  return true;
}

// The constants depend only on r: built once per r (bigint products and
// inverses), then copied.
bool make_const(int r, Oz2Const& c) {
  static std::mutex mu;
  static Oz2Const cache[OZ2_MAXR + 1];
  static bool ready[OZ2_MAXR + 1] = {false};
  if (r < 8 || r > OZ2_MAXR) return false;
  std::lock_guard<std::mutex> g(mu);
  if (!ready[r]) {
    if (!build_const(r, cache[r])) return false;
    ready[r] = true;
  }
  c = cache[r];
  return true;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
int round_up(int x, int q) { return ((x + q - 1) / q) * q; }

bool make_dims(int m, int n, int k, unsigned flags, Oz2Dims& d) {
  if (m < 0 || n < 0 || k < 0) return false;
  d.m = m;
  d.n = n;
  d.k = k;
  d.mp = round_up(std::max(m, 1), OZ2_TILE);
  d.np = round_up(std::max(n, 1), OZ2_TILE);
  d.kp = round_up(std::max(k, 1), OZ2_KPAD);
  d.cslabs = (d.kp + OZ2_CSLAB - 1) / OZ2_CSLAB;
  d.flags = flags;
  const double lim = 1099511627776.0;      // 2^40
  if ((double)d.mp * d.kp >= lim || (double)d.np * d.kp >= lim || (double)d.mp * d.np >= lim)
    return false;
  return true;
}

Oz2Layout make_layout(const Oz2Dims& d, const Oz2Const& c) {
  Oz2Layout L{};
  size_t o = 0;
  auto take = [&o](size_t bytes) { size_t at = o; o = align256(o + bytes); return at; };
  L.rowbits = take((size_t)d.mp * 8);
  L.colbits = take((size_t)d.np * 8);
  L.flagsA = take((size_t)d.mp * 4);
  L.flagsB = take((size_t)d.np * 4);
  L.Rmax = take((size_t)d.cslabs * d.mp * 4);
  L.Kmax = take((size_t)d.cslabs * d.np * 4);
  L.sA = take((size_t)d.mp * 4);
  L.tB = take((size_t)d.np * 4);
  L.eA = take((size_t)d.mp * 4);
  L.eB = take((size_t)d.np * 4);
  L.counters = take(64);
  L.listA = take((size_t)d.mp * 4);
  L.listB = take((size_t)d.np * 4);
  L.codesA = take((size_t)d.mp * d.kp);
  L.codesB = take((size_t)d.np * d.kp);
  L.etA = take((size_t)d.mp * (d.kp / 64) * 2);
  L.etB = take((size_t)d.np * (d.kp / 64) * 2);
  L.planesA = take((size_t)c.P * d.mp * d.kp);
  L.planesB = take((size_t)c.P * d.np * d.kp);
  L.tabs = take((size_t)c.tabsz * 4);
  // the fused route keeps the residues on chip, and its native fallback reads A
  // directly (no gathered panel)
  const bool fused = (d.flags & OZ2_FUSED) != 0;
  L.res = fused ? 0 : take((size_t)c.r * d.mp * d.np / 8 * 12);   // 12 bits per output
  L.panel = ((d.flags & OZ2_NO_FALLBACK) || fused)
                ? 0 : take((size_t)std::min(d.mp, OZ2_FBCAP) * d.k * 8);
  L.total = o;
  return L;
}

// ------------------------------------------------------------ batched GEMV
// Y = A X with X of nrhs <= 16 columns (the fused kernel of gemv.hip): k in
// chunks of 128, 128 rows of A per workgroup, and enough k-splits that every
// split spans at most 32768 k (exact FP32 accumulation) and the row blocks
// times the splits cover about 256 workgroups.
constexpr int kGemvRhs = 16, kGemvK = 128, kGemvRows = 128;

struct GemvShape {
  Oz2Dims d;          // n = nrhs, np = 16, mp = rows padded to 128, kp to 128
  int chunks, splits;
};

bool gemv_shape(int m, int k, int nrhs, unsigned flags, GemvShape& g) {
  if (m < 0 || k < 0 || nrhs < 0 || nrhs > kGemvRhs) return false;
  Oz2Dims& d = g.d;
  d.m = m;
  d.n = nrhs;
  d.k = k;
  d.mp = round_up(std::max(m, 1), kGemvRows);
  d.np = kGemvRhs;
  d.kp = round_up(std::max(k, 1), kGemvK);
  d.cslabs = 1;
  d.flags = flags | OZ2_SCALE_FIXED;
  if ((double)d.mp * d.kp >= 1099511627776.0) return false;
  g.chunks = d.kp / kGemvK;
  const int need = (g.chunks + 255) / 256;
  const int blocks = d.mp / kGemvRows;
  const int fill = std::min(g.chunks, (256 + blocks - 1) / blocks);
  g.splits = std::max(need, fill);
  return true;
}

Oz2Layout make_gemv_layout(const GemvShape& g, const Oz2Const& c) {
  const Oz2Dims& d = g.d;
  Oz2Layout L{};
  size_t o = 0;
  auto take = [&o](size_t bytes) { size_t at = o; o = align256(o + bytes); return at; };
  L.rowbits = take((size_t)d.mp * 8);
  L.colbits = take((size_t)d.np * 8);
  L.flagsA = take((size_t)d.mp * 4);
  L.flagsB = take((size_t)d.np * 4);
  L.Rmax = take((size_t)d.mp * 4);
  L.Kmax = take((size_t)d.np * 4);
  L.sA = take((size_t)d.mp * 4);
  L.tB = take((size_t)d.np * 4);
  L.eA = take((size_t)d.mp * 4);
  L.eB = take((size_t)d.np * 4);
  L.counters = take(64);
  L.listA = take((size_t)d.mp * 4);
  L.listB = take((size_t)d.np * 4);
  L.tabs = take((size_t)c.tabsz * 4);
  L.xfrag = take((size_t)g.chunks * c.P * 2048);
  L.part = take((size_t)g.splits * c.r * d.mp * kGemvRhs * 2);
  L.total = o;
  return L;
}

const unsigned kGemvFlags =
    OZ2_QUANT_TZ | OZ2_NO_FALLBACK | OZ2_FORCE_FALLBACK | OZ2_REUSE_A_SCALES;

const unsigned kKnownFlags = OZ2_ACCUMULATE | OZ2_SCALE_FIXED | OZ2_QUANT_TZ | OZ2_NO_FALLBACK |
                             OZ2_FORCE_FALLBACK | OZ2_KEEP_RESIDUES | OZ2_TIME_STAGES | OZ2_FUSED;

// The fused residue-GEMM + reconstruction kernel holds r <= 12 residues per
// output packed in four words and runs one exact FP32 slab of k.
bool fused_ok(const Oz2Dims& d, const Oz2Const& c) { return c.r <= 12 && d.kp <= OZ2_KSLAB; }

// The route of ozaki2_dgemm / _ex / _static: the fused kernel only when the
// caller asks for it.  Measured on MI355X at 8192^2 and 16384^2 with k from
// 256 to 4096 it is 1.2-1.5x slower than the staged route (its 128 x 128
// tiles need twice the operand bytes per FLOP from L2, and its CRT epilogue
// leaves the matrix cores idle), although it moves a fraction of the HBM
// bytes; the staged route stays the default.
unsigned route_flags(int, int, int, int, unsigned flags) { return flags; }

}  // namespace

int oz2_device_cus() {
  static const int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      return 256;
    return n;
  }();
  return cus;
}

namespace {

// gfx950 check, cached per device
int device_ok() {
  static std::mutex mu;
  static int cache[64];
  static bool init = false;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return OZ2_E_DEVICE;
  std::lock_guard<std::mutex> g(mu);
  if (!init) { for (int& x : cache) x = 0; init = true; }
  if (dev < 0 || dev >= 64) return OZ2_E_DEVICE;
  if (cache[dev] == 0) {
    hipDeviceProp_t p;
    if (hipGetDeviceProperties(&p, dev) != hipSuccess) return OZ2_E_DEVICE;
    cache[dev] = (std::strncmp(p.gcnArchName, "gfx950", 6) == 0) ? 1 : 2;
  }
  return cache[dev] == 1 ? OZ2_OK : OZ2_E_UNSUPPORTED;
}

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  uintptr_t a0 = (uintptr_t)a, a1 = a0 + abytes, b0 = (uintptr_t)b, b1 = b0 + bbytes;
  return a0 < b1 && b0 < a1;
}

size_t span_bytes(int rows, int cols, int ld) {
  if (rows <= 0 || cols <= 0) return 0;
  return ((size_t)(cols - 1) * ld + rows) * sizeof(double);
}

int check_mats(int m, int n, int k, const double* A, int lda, const double* B, int ldb,
               const double* C, int ldc) {
  if (m < 0 || n < 0 || k < 0) return OZ2_E_INVALID;
  if (lda < std::max(1, m) || ldb < std::max(1, k) || ldc < std::max(1, m)) return OZ2_E_INVALID;
  if (m > 0 && n > 0) {
    if (!C) return OZ2_E_INVALID;
    if (k > 0 && (!A || !B)) return OZ2_E_INVALID;
    size_t cb = span_bytes(m, n, ldc);
    if (k > 0 && (overlaps(C, cb, A, span_bytes(m, k, lda)) ||
                  overlaps(C, cb, B, span_bytes(k, n, ldb))))
      return OZ2_E_INVALID;
  }
  return OZ2_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? OZ2_OK : OZ2_E_DEVICE; }

}  // namespace

// ---------------------------------------------------------------- static scratch
// The workspace of ozaki2_dgemm_static: a file-scope device array, one copy on
// every GPU the library runs on, held until the process ends.  Host code never
// uses the array's name as an address (on the host it is only a stand-in for
// the device symbol): the device address of each GPU's copy comes from
// hipGetSymbolAddress, once per device, and is kept in g_scratch_ptr.
static __device__ __align__(256) uint8_t scratch[OZ2_STATIC_SCRATCH_BYTES];

// ------------------------------------------------------------------ plans
// Stage events of an OZ2_TIME_STAGES plan: 0 deconstruct start, 1 after scan +
// codes, 2 after the max-magnitude GEMM, 3 after the split, 4 / 5 around the
// residue GEMMs, 6 reconstruction start, 7 after it, 8 after the fallback.
constexpr int kStageEvents = 9;

struct ozaki2_plan_s {
  Oz2Dims d;
  Oz2Const c;
  Oz2Layout L;
  uint8_t* ws = nullptr;
  const double* A = nullptr;
  const double* B = nullptr;
  int lda = 0, ldb = 0;
  int stage = 0;      // 0 created, 1 deconstructed, 2 residues ready, 3 reconstructed
  int sides = 0;      // operands whose planes are in the workspace (OZ2_SIDE_A | OZ2_SIDE_B)
  bool tables = false;   // residue -> plane-byte tables built in the workspace (they depend on r only)
  hipEvent_t ev[kStageEvents] = {};
  bool timed = false;    // OZ2_TIME_STAGES: ev[] exist
  unsigned recorded = 0; // events recorded since the last deconstruct (bit i: ev[i])
};

namespace {

// records stage event i of a timed plan on stream s (no-op otherwise)
hipError_t mark(ozaki2_plan_s& p, int i, hipStream_t s) {
  if (!p.timed) return hipSuccess;
  const hipError_t e = hipEventRecord(p.ev[i], s);
  if (e == hipSuccess) p.recorded |= 1u << i;
  return e;
}

// Phase 1 for the operands in `side` (OZ2_SIDE_A, OZ2_SIDE_B or both).  One
// operand alone only under OZ2_SCALE_FIXED, where its scales do not depend on
// the other operand (no max-magnitude pass).
int run_deconstruct(ozaki2_plan_s& p, int side, hipStream_t s) {
  const Oz2Dims& d = p.d;
  // Each operand is read once for its scan and code bytes (one kernel), and
  // both operands are split in one launch, B's tiles first, so that the
  // second read finds B (read last) still in the 256 MiB memory-side cache.
  const bool codes = !(d.flags & OZ2_SCALE_FIXED);
  p.recorded = 0;
  hipError_t e = mark(p, 0, s);
  if (e == hipSuccess) e = oz2_launch_init(d, p.L, p.ws, side, s);
  for (int one : {OZ2_SIDE_A, OZ2_SIDE_B}) {
    if (!(side & one) || e != hipSuccess) continue;
    e = codes ? oz2_launch_scan_codes(d, p.L, p.ws, p.A, p.lda, p.B, p.ldb, one, s)
              : oz2_launch_scan(d, p.L, p.ws, p.A, p.lda, p.B, p.ldb, one, s);
  }
  if (codes && e == hipSuccess) e = oz2_launch_rebase(d, p.L, p.ws, side, s);
  if (e == hipSuccess) e = mark(p, 1, s);
  if (codes && e == hipSuccess) e = oz2_launch_codegemm(d, p.L, p.ws, s);
  if (e == hipSuccess) e = mark(p, 2, s);
  if (e == hipSuccess) e = oz2_launch_scales(d, p.L, p.c, p.ws, side, s);
  if (e == hipSuccess && !p.tables) {
    e = oz2_launch_tables(p.L, p.c, p.ws, s);
    p.tables = e == hipSuccess;
  }
  if (e == hipSuccess) e = oz2_launch_split(d, p.L, p.c, p.ws, p.A, p.lda, p.B, p.ldb, side, s);
  if (e == hipSuccess) e = mark(p, 3, s);
  return hip_status(e);
}

int run_reconstruct(ozaki2_plan_s& p, double* C, int ldc, hipStream_t s) {
  const bool fused = (p.d.flags & OZ2_FUSED) != 0;
  hipError_t e = mark(p, 6, s);
  if (e == hipSuccess)
    e = fused ? oz2_launch_fused(p.d, p.L, p.c, p.ws, C, ldc, s)
              : oz2_launch_reconstruct(p.d, p.L, p.c, p.ws, p.A, p.lda, C, ldc, s);
  if (e == hipSuccess) e = mark(p, 7, s);
  if (e == hipSuccess && !(p.d.flags & OZ2_NO_FALLBACK))
    e = fused ? oz2_launch_fallback_direct(p.d, p.L, p.ws, p.A, p.lda, p.B, p.ldb, C, ldc, s)
              : oz2_launch_fallback(p.d, p.L, p.ws, p.A, p.lda, p.B, p.ldb, C, ldc, s);
  if (e == hipSuccess) e = mark(p, 8, s);
  return hip_status(e);
}

// internal grow-only workspace of ozaki2_dgemm, per device.  Callers hold
// g_pool_mu from pool_get until their work is enqueued: a grow synchronises
// the device before it frees the old buffer, so work enqueued under the lock
// has finished with it by then, whichever thread grows the pool next.
struct Pool {
  void* ptr = nullptr;
  size_t bytes = 0;
};
std::mutex g_pool_mu;
Pool g_pool[64];

int pool_get(size_t need, void** out) {   // g_pool_mu held by the caller
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return OZ2_E_DEVICE;
  Pool& P = g_pool[dev];
  if (P.bytes < need) {
    if (P.ptr) {
      if (hipDeviceSynchronize() != hipSuccess) return OZ2_E_DEVICE;
      (void)hipFree(P.ptr);
      P.ptr = nullptr;
      P.bytes = 0;
    }
    size_t grow = std::max(need, (size_t)1 << 20);
    if (hipMalloc(&P.ptr, grow) != hipSuccess) {
      (void)hipGetLastError();
      P.ptr = nullptr;
      return OZ2_E_NOMEM;
    }
    P.bytes = grow;
  }
  *out = P.ptr;
  return OZ2_OK;
}

std::mutex g_scratch_mu;
void* g_scratch_ptr[64];

int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return OZ2_E_DEVICE;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return OZ2_E_DEVICE;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return OZ2_OK;
}

}  // namespace

extern "C" {

const char* ozaki2_status_string(int status) {
  switch (status) {
    case OZ2_OK: return "ok";
    case OZ2_E_INVALID: return "invalid argument";
    case OZ2_E_NOMEM: return "out of device memory";
    case OZ2_E_DEVICE: return "HIP runtime or launch error";
    case OZ2_E_UNSUPPORTED: return "unsupported device (gfx950 required)";
    case OZ2_E_WORKSPACE: return "workspace missing or too small";
    default: return "unknown status";
  }
}

int ozaki2_moduli(int num_moduli, int* host_out) {
  Oz2Const c;
  if (!host_out || !make_const(num_moduli, c)) return OZ2_E_INVALID;
  for (int i = 0; i < num_moduli; ++i) host_out[i] = c.m[i];
  return OZ2_OK;
}

// C = A B with at most 16 columns under the fixed scaling: ozaki2_dgemm_ex
// runs the fused GEMV of Alg. 2 (A deconstructed on the fly, fused mode F for
// tall-skinny products), whose results equal the staged fixed-scale path's
// bit for bit; plans always take the staged path.
static bool skinny_route(int n, unsigned flags) {
  return (flags & OZ2_SCALE_FIXED) && n <= kGemvRhs &&
         !(flags & (OZ2_ACCUMULATE | OZ2_FUSED | OZ2_KEEP_RESIDUES | OZ2_TIME_STAGES));
}

size_t ozaki2_workspace_bytes(int m, int n, int k, int num_moduli, unsigned flags) {
  Oz2Const c;
  Oz2Dims d;
  if ((flags & ~kKnownFlags) || !make_const(num_moduli, c) || !make_dims(m, n, k, flags, d))
    return 0;
  const size_t staged = make_layout(d, c).total;
  if (!skinny_route(n, flags)) return staged;
  // enough for either route: the same size serves ozaki2_plan_create
  return std::max(staged, ozaki2_gemv_workspace_bytes(m, k, n, num_moduli));
}

int ozaki2_plan_create(ozaki2_plan_t* out, int m, int n, int k, int num_moduli, unsigned flags,
                       void* workspace, size_t ws_bytes) {
  if (!out) return OZ2_E_INVALID;
  *out = nullptr;
  if (flags & ~kKnownFlags) return OZ2_E_INVALID;
  if (m <= 0 || n <= 0 || k <= 0) return OZ2_E_INVALID;
  ozaki2_plan_s* p = new (std::nothrow) ozaki2_plan_s();
  if (!p) return OZ2_E_NOMEM;
  if (!make_const(num_moduli, p->c) || !make_dims(m, n, k, flags, p->d) ||
      ((flags & OZ2_FUSED) && (flags & OZ2_KEEP_RESIDUES))) {
    delete p;
    return OZ2_E_INVALID;
  }
  if ((flags & OZ2_FUSED) && !fused_ok(p->d, p->c)) {
    delete p;
    return OZ2_E_UNSUPPORTED;
  }
  p->L = make_layout(p->d, p->c);
  if (!workspace || ws_bytes < p->L.total || ((uintptr_t)workspace & 255)) {
    delete p;
    return OZ2_E_WORKSPACE;
  }
  int st = device_ok();
  if (st != OZ2_OK) {
    delete p;
    return st;
  }
  if (flags & OZ2_TIME_STAGES) {
    for (int i = 0; i < kStageEvents; ++i) {
      if (hipEventCreate(&p->ev[i]) != hipSuccess) {
        for (int j = 0; j < i; ++j) (void)hipEventDestroy(p->ev[j]);
        delete p;
        return OZ2_E_DEVICE;
      }
    }
    p->timed = true;
  }
  p->ws = (uint8_t*)workspace;
  *out = p;
  return OZ2_OK;
}

int ozaki2_plan_destroy(ozaki2_plan_t plan) {
  if (plan && plan->timed)
    for (int i = 0; i < kStageEvents; ++i) (void)hipEventDestroy(plan->ev[i]);
  delete plan;
  return OZ2_OK;
}

int ozaki2_deconstruct(ozaki2_plan_t p, const double* A, int lda, const double* B, int ldb,
                       void* stream) {
  if (!p || !A || !B) return OZ2_E_INVALID;
  if (lda < std::max(1, p->d.m) || ldb < std::max(1, p->d.k)) return OZ2_E_INVALID;
  p->A = A;
  p->B = B;
  p->lda = lda;
  p->ldb = ldb;
  int st = run_deconstruct(*p, OZ2_SIDE_A | OZ2_SIDE_B, (hipStream_t)stream);
  p->sides = st == OZ2_OK ? (OZ2_SIDE_A | OZ2_SIDE_B) : 0;
  p->stage = st == OZ2_OK ? 1 : 0;
  return st;
}

namespace {
// Operand-stationary use: re-deconstruct one operand, keep the other's planes.
int deconstruct_one(ozaki2_plan_t p, int side, const double* X, int ld, void* stream) {
  if (!p || !X || !(p->d.flags & OZ2_SCALE_FIXED)) return OZ2_E_INVALID;
  if (ld < std::max(1, side == OZ2_SIDE_A ? p->d.m : p->d.k)) return OZ2_E_INVALID;
  if (side == OZ2_SIDE_A) {
    p->A = X;
    p->lda = ld;
  } else {
    p->B = X;
    p->ldb = ld;
  }
  p->sides &= ~side;
  int st = run_deconstruct(*p, side, (hipStream_t)stream);
  if (st == OZ2_OK) p->sides |= side;
  p->stage = (st == OZ2_OK && p->sides == (OZ2_SIDE_A | OZ2_SIDE_B)) ? 1 : 0;
  return st;
}
}  // namespace

int ozaki2_deconstruct_a(ozaki2_plan_t p, const double* A, int lda, void* stream) {
  return deconstruct_one(p, OZ2_SIDE_A, A, lda, stream);
}

int ozaki2_deconstruct_b(ozaki2_plan_t p, const double* B, int ldb, void* stream) {
  return deconstruct_one(p, OZ2_SIDE_B, B, ldb, stream);
}

int ozaki2_residue_gemm(ozaki2_plan_t p, void* stream) {
  if (!p || p->stage < 1) return OZ2_E_INVALID;
  const hipStream_t s = (hipStream_t)stream;
  hipError_t e = mark(*p, 4, s);
  // a fused plan runs its residue GEMMs inside the reconstruction
  if (e == hipSuccess && !(p->d.flags & OZ2_FUSED))
    e = oz2_launch_resgemm(p->d, p->L, p->c, p->ws, s);
  if (e == hipSuccess) e = mark(*p, 5, s);
  int st = hip_status(e);
  if (st == OZ2_OK) p->stage = 2;
  return st;
}

int ozaki2_reconstruct(ozaki2_plan_t p, double* C, int ldc, void* stream) {
  if (!p || p->stage < 2 || !C || ldc < std::max(1, p->d.m)) return OZ2_E_INVALID;
  int st = check_mats(p->d.m, p->d.n, p->d.k, p->A, p->lda, p->B, p->ldb, C, ldc);
  if (st != OZ2_OK) return st;
  st = run_reconstruct(*p, C, ldc, (hipStream_t)stream);
  if (st == OZ2_OK) p->stage = 3;
  return st;
}

int ozaki2_dgemm_ex(int m, int n, int k, const double* A, int lda, const double* B, int ldb,
                    double* C, int ldc, int num_moduli, unsigned flags, void* workspace,
                    size_t ws_bytes, void* stream) {
  if ((flags & ~kKnownFlags) || (flags & OZ2_TIME_STAGES)) return OZ2_E_INVALID;
  if (num_moduli < 8 || num_moduli > OZ2_MAXR) return OZ2_E_INVALID;
  int st = check_mats(m, n, k, A, lda, B, ldb, C, ldc);
  if (st != OZ2_OK) return st;
  if (m == 0 || n == 0) return OZ2_OK;
  st = device_ok();
  if (st != OZ2_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if (k == 0) {
    if (flags & OZ2_ACCUMULATE) return OZ2_OK;
    return hip_status(oz2_launch_fill(C, m, n, ldc, s));
  }
  if (skinny_route(n, flags))
    return ozaki2_gemv_batched(m, k, n, A, lda, B, ldb, C, ldc, num_moduli, flags & kGemvFlags,
                               workspace, ws_bytes, stream);
  ozaki2_plan_s p;
  flags = route_flags(m, n, k, num_moduli, flags);
  if (!make_const(num_moduli, p.c) || !make_dims(m, n, k, flags, p.d)) return OZ2_E_INVALID;
  if ((flags & OZ2_FUSED) && ((flags & OZ2_KEEP_RESIDUES) || !fused_ok(p.d, p.c)))
    return (flags & OZ2_KEEP_RESIDUES) ? OZ2_E_INVALID : OZ2_E_UNSUPPORTED;
  p.L = make_layout(p.d, p.c);
  if (!workspace || ws_bytes < p.L.total || ((uintptr_t)workspace & 255)) return OZ2_E_WORKSPACE;
  p.ws = (uint8_t*)workspace;
  p.A = A;
  p.B = B;
  p.lda = lda;
  p.ldb = ldb;
  st = run_deconstruct(p, OZ2_SIDE_A | OZ2_SIDE_B, s);
  if (st != OZ2_OK) return st;
  if (!(flags & OZ2_FUSED)) {
    st = hip_status(oz2_launch_resgemm(p.d, p.L, p.c, p.ws, s));
    if (st != OZ2_OK) return st;
  }
  return run_reconstruct(p, C, ldc, s);
}

int ozaki2_dgemm(int m, int n, int k, const double* A, int lda, const double* B, int ldb,
                 double* C, int ldc, int num_moduli, void* stream) {
  if (num_moduli < 8 || num_moduli > OZ2_MAXR) return OZ2_E_INVALID;
  int st = check_mats(m, n, k, A, lda, B, ldb, C, ldc);
  if (st != OZ2_OK) return st;
  if (m == 0 || n == 0) return OZ2_OK;
  size_t need = ozaki2_workspace_bytes(m, n, k, num_moduli, route_flags(m, n, k, num_moduli, 0));
  if (need == 0) return OZ2_E_INVALID;
  st = device_ok();
  if (st != OZ2_OK) return st;
  std::lock_guard<std::mutex> g(g_pool_mu);
  void* ws = nullptr;
  st = pool_get(need, &ws);
  if (st != OZ2_OK) return st;
  return ozaki2_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, num_moduli, 0, ws, need, stream);
}

int ozaki2_dgemm_static(int m, int n, int k, const double* A, int lda, const double* B, int ldb,
                        double* C, int ldc, int num_moduli, void* stream) {
  if (num_moduli < 8 || num_moduli > OZ2_MAXR) return OZ2_E_INVALID;
  int st = check_mats(m, n, k, A, lda, B, ldb, C, ldc);
  if (st != OZ2_OK) return st;
  if (m == 0 || n == 0) return OZ2_OK;
  const size_t need = ozaki2_workspace_bytes(m, n, k, num_moduli, 0);
  if (need == 0) return OZ2_E_INVALID;
  if (need > OZ2_STATIC_SCRATCH_BYTES) return OZ2_E_WORKSPACE;
  st = device_ok();
  if (st != OZ2_OK) return st;
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != OZ2_OK) return st;
  // every kernel of the staged path clears what it accumulates into (k_init)
  // and rebuilds the plane tables, so the previous call's contents do not matter
  return ozaki2_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, num_moduli, 0, ws, need, stream);
}

int ozaki2_dgemm_strided_batched(int m, int n, int k, const double* A, int lda, long long strideA,
                                 const double* B, int ldb, long long strideB, double* C, int ldc,
                                 long long strideC, int batch, int num_moduli, void* stream) {
  if (batch < 0 || num_moduli < 8 || num_moduli > OZ2_MAXR) return OZ2_E_INVALID;
  if (strideA < 0 || strideB < 0 || strideC < 0) return OZ2_E_INVALID;
  int st = check_mats(m, n, k, A, lda, B, ldb, C, ldc);
  if (st != OZ2_OK) return st;
  if (batch == 0 || m == 0 || n == 0) return OZ2_OK;
  if (batch > 1 && (size_t)strideC * sizeof(double) < span_bytes(m, n, ldc)) return OZ2_E_INVALID;
  if (m <= 64 && n <= 64 && k <= 64 && k > 0) {
    // one launch for all problems: every stage inside one workgroup per problem
    Oz2Const c;
    if (!make_const(num_moduli, c)) return OZ2_E_INVALID;
    st = device_ok();
    if (st != OZ2_OK) return st;
    std::lock_guard<std::mutex> g(g_pool_mu);
    void* ws = nullptr;
    st = pool_get(align256((size_t)c.tabsz * 4), &ws);
    if (st != OZ2_OK) return st;
    Oz2Layout L{};
    L.tabs = 0;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = oz2_launch_tables(L, c, (uint8_t*)ws, s);
    if (e == hipSuccess)
      e = oz2_launch_batched(c, m, n, k, batch, A, lda, strideA, B, ldb, strideB, C, ldc, strideC,
                             (const uint32_t*)ws, nullptr, s);
    return e == hipSuccess ? OZ2_OK : OZ2_E_DEVICE;
  }
  size_t need = ozaki2_workspace_bytes(m, n, k, num_moduli, 0);
  if (need == 0) return OZ2_E_INVALID;
  st = device_ok();
  if (st != OZ2_OK) return st;
  std::lock_guard<std::mutex> g(g_pool_mu);
  void* ws = nullptr;
  st = pool_get(need, &ws);
  if (st != OZ2_OK) return st;
  for (int b = 0; b < batch; ++b) {
    st = ozaki2_dgemm_ex(m, n, k, A + (size_t)b * strideA, lda, B + (size_t)b * strideB, ldb,
                         C + (size_t)b * strideC, ldc, num_moduli, 0, ws, need, stream);
    if (st != OZ2_OK) return st;
  }
  return OZ2_OK;
}

size_t ozaki2_gemv_workspace_bytes(int m, int k, int nrhs, int num_moduli) {
  Oz2Const c;
  GemvShape g;
  if (!make_const(num_moduli, c) || !gemv_shape(m, k, nrhs, 0, g)) return 0;
  return make_gemv_layout(g, c).total;
}

int ozaki2_gemv_batched(int m, int k, int nrhs, const double* A, int lda, const double* X, int ldx,
                        double* Y, int ldy, int num_moduli, unsigned flags, void* workspace,
                        size_t ws_bytes, void* stream) {
  if (flags & ~kGemvFlags) return OZ2_E_INVALID;
  if (num_moduli < 8 || num_moduli > OZ2_MAXR || nrhs > kGemvRhs) return OZ2_E_INVALID;
  int st = check_mats(m, nrhs, k, A, lda, X, ldx, Y, ldy);
  if (st != OZ2_OK) return st;
  if (m == 0 || nrhs == 0) return OZ2_OK;
  hipStream_t s = (hipStream_t)stream;
  if (k == 0) {
    st = device_ok();
    return st != OZ2_OK ? st : hip_status(oz2_launch_fill(Y, m, nrhs, ldy, s));
  }
  Oz2Const c;
  GemvShape g;
  if (!make_const(num_moduli, c) || !gemv_shape(m, k, nrhs, flags, g)) return OZ2_E_INVALID;
  // the fused kernel treats moduli r-6 .. r-1 (the six squares) as square
  for (int i = 0; i < c.r; ++i)
    if ((c.sq[i] != 0) != (i >= c.r - 6)) return OZ2_E_UNSUPPORTED;
  const Oz2Layout L = make_gemv_layout(g, c);
  if (!workspace || ws_bytes < L.total || ((uintptr_t)workspace & 255)) return OZ2_E_WORKSPACE;
  st = device_ok();
  if (st != OZ2_OK) return st;
  uint8_t* ws = (uint8_t*)workspace;
  const Oz2Dims& d = g.d;
  const unsigned tz = (flags & OZ2_QUANT_TZ) ? 1u : 0u;
  const int listed = (flags & OZ2_FORCE_FALLBACK) ? 1 : 0;
  // with OZ2_REUSE_A_SCALES, A's side (scales, flags, list, counter) and the
  // plane tables are the previous call's
  const bool reuse = (flags & OZ2_REUSE_A_SCALES) != 0;
  const int sides = reuse ? OZ2_SIDE_B : (OZ2_SIDE_A | OZ2_SIDE_B);
  hipError_t e = oz2_launch_init(d, L, ws, sides, s);
  if (e == hipSuccess) e = oz2_launch_scan(d, L, ws, A, lda, X, ldx, sides, s);
  if (e == hipSuccess) e = oz2_launch_scales(d, L, c, ws, sides, s);
  if (e == hipSuccess && !reuse) e = oz2_launch_tables(L, c, ws, s);
  if (e == hipSuccess)
    e = oz2_launch_gemv_xplanes(c, X, ldx, k, nrhs, (const int32_t*)(ws + L.tB),
                                (uint32_t*)(ws + L.flagsB), (int*)(ws + L.counters) + 1,
                                (int*)(ws + L.listB), listed, (const uint32_t*)(ws + L.tabs), tz,
                                ws + L.xfrag, s);
  if (e == hipSuccess)
    e = oz2_launch_gemv(c, A, lda, m, k, g.splits, (const int32_t*)(ws + L.sA),
                        (uint32_t*)(ws + L.flagsA), (int*)(ws + L.counters), (int*)(ws + L.listA),
                        listed, ws + L.xfrag, (const uint32_t*)(ws + L.tabs), tz,
                        (int16_t*)(ws + L.part), d.mp, s);
  const int nofb = (flags & OZ2_NO_FALLBACK) ? 1 : 0;
  if (e == hipSuccess)
    e = oz2_launch_gemv_crt(c, (const int16_t*)(ws + L.part), g.splits, d.mp, m, nrhs,
                            (const int32_t*)(ws + L.sA), (const int32_t*)(ws + L.tB),
                            (const uint32_t*)(ws + L.flagsA), (const uint32_t*)(ws + L.flagsB),
                            nofb, Y, ldy, s);
  if (e == hipSuccess && !nofb) e = oz2_launch_fallback_direct(d, L, ws, A, lda, X, ldx, Y, ldy, s);
  return hip_status(e);
}

void ozaki2_finalize(void) {
  std::lock_guard<std::mutex> g(g_pool_mu);
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess) return;
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (int d = 0; d < ndev && d < 64; ++d) {
    if (!g_pool[d].ptr) continue;
    if (hipSetDevice(d) == hipSuccess) {
      (void)hipDeviceSynchronize();
      (void)hipFree(g_pool[d].ptr);
    }
    g_pool[d].ptr = nullptr;
    g_pool[d].bytes = 0;
  }
  (void)hipSetDevice(cur);
}

size_t ozaki2_plan_query_bytes(ozaki2_plan_t p, int what) {
  if (!p) return 0;
  const size_t m = p->d.m, n = p->d.n, k = p->d.k;
  switch (what) {
    case OZ2_Q_EXPONENTS: return (m + n) * 4;
    case OZ2_Q_MAXIMA: return (m + n) * 8;
    case OZ2_Q_SCALES: return (m + n) * 4;
    case OZ2_Q_FLAGS: return (m + n) * 4;
    case OZ2_Q_CODES: return (m + n) * k;
    case OZ2_Q_PLANES: return (size_t)p->c.P * (m + n) * k;
    case OZ2_Q_RESIDUES: return (size_t)p->c.r * m * n * 2;
    case OZ2_Q_INTEGERS: return m * n * OZ2_NLIMB * 4;
    case OZ2_Q_FALLBACK_COUNT: return 8;
    case OZ2_Q_STAGE_TIMES: return 6 * sizeof(float);
    default: return 0;
  }
}

int ozaki2_plan_query(ozaki2_plan_t p, int what, void* host_out, size_t bytes) {
  if (!p || !host_out) return OZ2_E_INVALID;
  const size_t need = ozaki2_plan_query_bytes(p, what);
  if (need == 0 || bytes < need) return OZ2_E_INVALID;
  const bool residues = what == OZ2_Q_RESIDUES || what == OZ2_Q_INTEGERS;
  if (p->stage < (residues ? 2 : 1)) return OZ2_E_INVALID;
  if (residues && (p->d.flags & OZ2_FUSED)) return OZ2_E_INVALID;   // never materialised
  if (hipDeviceSynchronize() != hipSuccess) return OZ2_E_DEVICE;
  const Oz2Dims& d = p->d;
  const Oz2Layout& L = p->L;
  uint8_t* ws = p->ws;
  uint8_t* out = (uint8_t*)host_out;
  auto cp = [](void* dst, const void* src, size_t b) {
    return hipMemcpy(dst, src, b, hipMemcpyDeviceToHost) == hipSuccess;
  };
  switch (what) {
    case OZ2_Q_EXPONENTS:
      if (!cp(out, ws + L.eA, (size_t)d.m * 4) || !cp(out + (size_t)d.m * 4, ws + L.eB, (size_t)d.n * 4))
        return OZ2_E_DEVICE;
      return OZ2_OK;
    case OZ2_Q_MAXIMA: {
      std::vector<uint32_t> R((size_t)d.cslabs * d.mp), K((size_t)d.cslabs * d.np);
      if (!cp(R.data(), ws + L.Rmax, R.size() * 4) || !cp(K.data(), ws + L.Kmax, K.size() * 4))
        return OZ2_E_DEVICE;
      uint64_t* o = (uint64_t*)out;
      for (int i = 0; i < d.m; ++i) {
        uint64_t s = 0;
        for (int sl = 0; sl < d.cslabs; ++sl) s += R[(size_t)sl * d.mp + i];
        o[i] = s;
      }
      for (int j = 0; j < d.n; ++j) {
        uint64_t s = 0;
        for (int sl = 0; sl < d.cslabs; ++sl) s += K[(size_t)sl * d.np + j];
        o[d.m + j] = s;
      }
      return OZ2_OK;
    }
    case OZ2_Q_SCALES:
      if (!cp(out, ws + L.sA, (size_t)d.m * 4) || !cp(out + (size_t)d.m * 4, ws + L.tB, (size_t)d.n * 4))
        return OZ2_E_DEVICE;
      return OZ2_OK;
    case OZ2_Q_FLAGS:
      if (!cp(out, ws + L.flagsA, (size_t)d.m * 4) ||
          !cp(out + (size_t)d.m * 4, ws + L.flagsB, (size_t)d.n * 4))
        return OZ2_E_DEVICE;
      return OZ2_OK;
    case OZ2_Q_CODES:
    case OZ2_Q_PLANES: {
      // K-blocked [kp/64][rows_pad][64] per plane -> [rows][k]
      const bool codes = what == OZ2_Q_CODES;
      const int P = codes ? 1 : p->c.P;
      size_t o = 0;
      for (int side = 0; side < 2; ++side) {
        const int rows = side ? d.n : d.m, rp = side ? d.np : d.mp;
        const size_t base = codes ? (side ? L.codesB : L.codesA) : (side ? L.planesB : L.planesA);
        std::vector<uint8_t> raw((size_t)rp * d.kp);
        for (int pl = 0; pl < P; ++pl) {
          if (!cp(raw.data(), ws + base + (size_t)pl * rp * d.kp, raw.size())) return OZ2_E_DEVICE;
          for (int rr = 0; rr < rows; ++rr)
            for (int l = 0; l < d.k; ++l)
              out[o + (size_t)rr * d.k + l] =
                  raw[((size_t)(l / OZ2_KBLK) * rp + rr) * OZ2_KBLK + (l % OZ2_KBLK)];
          o += (size_t)rows * d.k;
        }
      }
      return OZ2_OK;
    }
    case OZ2_Q_RESIDUES: {
      // [tile][wave 8][x 4][y 2] blocks of 384 words per modulus holding
      // each lane's 2 records of 3 words (word w of lane L at 6 L + w, or
      // pair-major at 128 (w / 2) + 2 L + w % 2: oz2_pair_records), output
      // 8h + e of a lane in slot e of record h, as x + floor(m/2) + 32 -> the
      // representative x itself, [r][n][m]
      const size_t plane = (size_t)d.mp * d.np / 8 * 3;
      std::vector<uint32_t> raw((size_t)p->c.r * plane);
      if (!cp(raw.data(), ws + L.res, raw.size() * 4)) return OZ2_E_DEVICE;
      int16_t* o = (int16_t*)out;
      const int ntm = d.mp / OZ2_TILE;
      const bool pair = oz2_pair_records(d);
      for (int i = 0; i < p->c.r; ++i)
        for (size_t t = 0; t < (size_t)d.mp * d.np / 16; ++t) {
          const size_t tile = t >> 12;
          const int q = (int)(t & 4095), lane = q & 63, blk = q >> 6;
          const int y = blk & 1, x = (blk >> 1) & 3, w = blk >> 3;
          const int tm = (int)(tile % ntm), tn = (int)(tile / ntm);
          const int row = tm * OZ2_TILE + (w >> 2) * 128 + 32 * x + 4 * (lane >> 5);
          const int col = tn * OZ2_TILE + (w & 3) * 64 + 32 * y + (lane & 31);
          if (col >= d.n) continue;
          const uint32_t* blkw = raw.data() + (size_t)i * plane + (t >> 6) * 384;
          uint32_t rec[6];
          for (int w = 0; w < 6; ++w)
            rec[w] = blkw[pair ? 128 * (w / 2) + 2 * lane + w % 2 : 6 * lane + w];
          for (int e = 0; e < 16; ++e) {
            const int rr = row + 8 * (e >> 2) + (e & 3);
            if (rr >= d.m) continue;
            const int bit = 96 * (e >> 3) + 12 * (e & 7);
            const uint64_t two = (uint64_t)rec[bit >> 5] |
                                 ((bit >> 5) + 1 < 6 ? (uint64_t)rec[(bit >> 5) + 1] << 32 : 0);
            const int u = (int)((two >> (bit & 31)) & 0xFFFu);
            o[((size_t)i * d.n + col) * d.m + rr] = (int16_t)(u - (p->c.m[i] / 2 + 32));
          }
        }
      return OZ2_OK;
    }
    case OZ2_Q_INTEGERS: {
      uint32_t* dev = nullptr;
      if (hipMalloc(&dev, need) != hipSuccess) return OZ2_E_NOMEM;
      hipError_t e = oz2_launch_integers(d, L, p->c, ws, dev, nullptr);
      if (e == hipSuccess) e = hipDeviceSynchronize();
      if (e == hipSuccess) e = hipMemcpy(out, dev, need, hipMemcpyDeviceToHost);
      (void)hipFree(dev);
      return hip_status(e);
    }
    case OZ2_Q_FALLBACK_COUNT:
      return cp(out, ws + L.counters, 8) ? OZ2_OK : OZ2_E_DEVICE;
    case OZ2_Q_STAGE_TIMES: {
      if (!p->timed || p->recorded != (1u << kStageEvents) - 1u) return OZ2_E_INVALID;
      float* o = (float*)out;
      const int from[6] = {0, 1, 2, 4, 6, 7}, to[6] = {1, 2, 3, 5, 7, 8};
      for (int i = 0; i < 6; ++i)
        if (hipEventElapsedTime(&o[i], p->ev[from[i]], p->ev[to[i]]) != hipSuccess)
          return OZ2_E_DEVICE;
      return OZ2_OK;
    }
    default:
      return OZ2_E_INVALID;
  }
}

// ---------------------------------------------------------------- probes
// (include/ozaki2_probes.h; these two need the plan constants, the rest
// are in probes.hip)
int ozaki2_probe_crt(int num_moduli, const short* residues, const int* shifts, int n,
                     unsigned* words, double* rounded, void* stream) {
  Oz2Const c;
  if (n < 0 || !make_const(num_moduli, c)) return OZ2_E_INVALID;
  if (n > 0 && (!residues || !shifts || !words || !rounded)) return OZ2_E_INVALID;
  const int st = device_ok();
  if (st != OZ2_OK) return st;
  return hip_status(oz2_launch_crt_probe(c, (const int16_t*)residues, shifts, n, (uint32_t*)words,
                                         rounded, (hipStream_t)stream));
}

int ozaki2_probe_batched_integers(int m, int n, int k, const double* A, int lda,
                                  long long strideA, const double* B, int ldb, long long strideB,
                                  int batch, int num_moduli, unsigned* words, void* stream) {
  Oz2Const c;
  if (m < 1 || n < 1 || k < 1 || m > 64 || n > 64 || k > 64 || batch < 0) return OZ2_E_INVALID;
  if (lda < m || ldb < k || strideA < 0 || strideB < 0 || !make_const(num_moduli, c))
    return OZ2_E_INVALID;
  if (batch == 0) return OZ2_OK;
  if (!A || !B || !words) return OZ2_E_INVALID;
  int st = device_ok();
  if (st != OZ2_OK) return st;
  std::lock_guard<std::mutex> g(g_pool_mu);
  void* ws = nullptr;
  st = pool_get(align256((size_t)c.tabsz * 4), &ws);
  if (st != OZ2_OK) return st;
  Oz2Layout L{};
  L.tabs = 0;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = oz2_launch_tables(L, c, (uint8_t*)ws, s);
  // C is not written on this path (the kernel writes the integers instead)
  if (e == hipSuccess)
    e = oz2_launch_batched(c, m, n, k, batch, A, lda, strideA, B, ldb, strideB, nullptr, m, 0,
                           (const uint32_t*)ws, (uint32_t*)words, s);
  return hip_status(e);
}

}  // extern "C"
