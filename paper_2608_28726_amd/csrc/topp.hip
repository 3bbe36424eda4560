// Top-p (nucleus) features: the nucleus is the shortest prefix of the token
// order (larger logit first, equal logits by lower index) whose probability
// mass reaches P of the total, k = min{ j : C_j >= P * S }; the distribution
// features are then those of the renormalised nucleus (the per-token
// features of Pro-Router, Sec. 3.1, Eq. 3, after top-p truncation).
//
// One 512-thread workgroup per row, two reads of the row in the common case:
//  1. the stats pass of the row kernel (max M, rank of y, argmax, margin)
//     also builds a histogram in LDS: 4096 bins over the distance
//     (A0 - z) / T in [-25, 50) nats from an anchor A0, the workgroup's
//     largest logit among the first vectors (known before the pass
//     starts), each holding the count and the summed offsets of its logits
//     from the bin centre (fixed point), plus a list of the few logits more
//     than 25 nats above A0. A bin's mass is its count times the mass at
//     its centre, corrected to first order by the offsets (relative error
//     below 5e-5: bins are 0.018 nats wide); the prefix sums locate a window
//     of bins whose cumulative mass brackets P of the total with a relative
//     margin of 5e-4. (Integer LDS atomics are far cheaper than float ones);
//  2. a second pass that sums the masses above the window and in total and
//     gathers the window's logits into LDS, in one of three forms: sparse
//     (peaked rows: only the buckets that can reach the window are read, in
//     float64, and the mass below the window comes from the histogram with
//     a bound on its error); float32 (flat rows: every binned logit's mass
//     by the hardware exp2, float64 sums, and a certified bound on the
//     error of the test quantity); float64 over every binned logit (where
//     neither bound decides);
//  3. a bitonic sort of the window (descending; one wave in registers for
//     up to 512 logits) and a float64 scan along it give k; it is taken
//     only where the uncertainty of the sums leaves one index, and the
//     crossing is verified to lie inside the window. A larger window is
//     first split into 256 sub-buckets of its values with fixed-point sums
//     (integer atomics), and only the sub-buckets the crossing can fall in
//     are sorted.
// Logits beyond 50 nats can never be in a nucleus with P < 1 (their total
// mass is below V * e^-50 of S). Float64 exponentials use a table-driven
// method (Tang, ACM TOMS 15(2), 1989): exp(d) = 2^(n/64) * exp(r) with
// |r| <= ln2/128 and a degree-5 polynomial.
//
// When the histogram cannot be used (no finite anchor, an overfull list or
// window, or a crossing outside the window) the row falls back to the
// three-pass method: a 4096-bin float64 histogram relative to M, exact sums
// above the crossing bins with their logits gathered, sorted and scanned,
// and for overfull crossing bins a byte-wise radix refinement over
// order-preserving keys (four more reads, and one for exact sums above the
// boundary value) that resolves ties by counting.
#include "topp.h"

#include <type_traits>

#include "p2.h"
#include "row_scan.h"
#include "topk.h"

namespace pr {

using namespace scan;

namespace {

constexpr int kTpBlock = 512;
constexpr int kBins = 4096;     // fallback histogram: bins over kDMax nats below M
constexpr float kDMax = 50.0f;  // nats below the maximum
constexpr int kCap = 4096;      // gathered logits sorted in LDS
constexpr int kNW = kTpBlock / kWave;
constexpr int kSub = 256;  // sub-buckets of a window of more than 512 logits
constexpr int kHB = 4096;         // histogram bins of the stats pass
constexpr float kHAbove = 25.0f;  // nats above the anchor covered by the bins
constexpr float kHSpan = 75.0f;   // nats covered: [-kHAbove, kDMax)
constexpr float kHK = kHB / kHSpan;  // bins per nat
constexpr int kAboveCap = 512;    // logits above the bins, kept in a list
constexpr double kWinMargin = 5e-4;  // relative margin of the window around P * S
constexpr int kOffBits = 12;         // fixed-point bits of a logit's position inside its bin
constexpr float kOffQ = 4096.0f;     // 2^kOffBits
constexpr int kCountShift = 40;      // a histogram word: count << kCountShift | offset sum
constexpr double kLog2eD = 1.4426950408889634;  // log2(e)
constexpr double kLn2D = 0.6931471805599453;    // ln(2)
#ifndef PR_APPROX_LDX
#define PR_APPROX_LDX 4  // loads per lane in flight in the float32 pass
#endif
// Loads per lane in flight in the first pass and the float32 pass: bfloat16
// vectors hold 8 logits each, twice the registers of a float32 vector once
// unpacked; at a depth of 4 the bfloat16 kernel spilled about 40 registers
// and its top-p rows took 1.8 times as long.
template <typename Tin>
constexpr int first_pass_depth() { return sizeof(Tin) == 2 ? 2 : 4; }
template <typename Tin>
constexpr int approx_depth() { return sizeof(Tin) == 2 ? 2 : PR_APPROX_LDX; }
// Relative error bound of the hardware exp2 (v_exp_f32) for arguments in
// [-100, 1]; its largest error over every float there is 8.49e-8 (a GPU test
// re-checks the whole range).
constexpr double kExp2RelErr = 1.0e-7;
constexpr double kTSlack = 0.05;  // the float32 pass's frame: see approx_cut

struct TpShared {
  union {
    struct {
      double mass[kBins];
      uint32_t cnt[kBins];
    } lg;              // fallback histogram
    struct {
      // stats-pass histogram: per bin, the count (top 24 bits) and the
      // summed positions inside the bin (low 40 bits: each logit adds
      // floor((offset + 1/2) * kOffQ) in [0, kOffQ), so the field stays
      // below 2^40 while V < 2^24)
      uint64_t bins[kHB + 1];  // bins[kHB] takes the logits outside them (never read)
    } hs;
    double wtab[kHB];  // exact pass: exp of each bin centre's distance from M
  } u;
  float win[kCap];
  float above[kAboveCap];
  double exptab[64];  // 2^(j/64)
  double red_d[2][kNW];
  uint32_t red_u[kNW];
  uint32_t red_m[2][kNW];
  float red_f[kNW];
  float topk[topk::kMaxK];  // the row's K largest logits (sequence variant)
  double S64, target, massAbove, Eabove, SN, EN;
  uint32_t b_lo, b_hi, wcount, cntAbove, jfirst, rcount, n_above;
  int32_t hb_lo, hb_hi;
  int32_t active;
  Partial p;
  uint32_t fix;
  // per digit of the three-pass method's radix refinement, or per
  // sub-bucket of a large window's cut (never in use at the same time)
  union {
    struct {
      double mass[256], E[256];
      uint32_t cnt[256];
    } rx;
    struct {
      unsigned long long q[kSub];   // masses, fixed point
      unsigned long long qe[kSub];  // entropy terms, fixed point (two's complement)
      uint32_t cnt[kSub];
    } sb;
  } r;
  uint32_t prefix, rdigit;
  struct {
    double m, e, t_lo, t_hi;  // above the crossing sub-buckets; the widened thresholds
    uint32_t c, s_first, s_last;
  } sc;
  // the window location's per-wave exchanges (each slot written once per
  // row, so that no barrier has to follow a read)
  struct {
    double scan[kNW], sa[kNW], seg[kNW], d[2][kNW];
    uint32_t u[3][kNW];
  } loc;
};

// Calls fn(z) for every logit of the row (order irrelevant), with the
// double-buffered loop of the scan, LDX vector loads per lane in flight
// (lanes past the end see -inf, which every fn ignores).
template <typename Tin, int LDX = 2, typename Fn>
__device__ __forceinline__ void for_each_logit(const void* row, int32_t V, int64_t h, int64_t nvec, Fn fn) {
  constexpr int VEC = Elem<Tin>::kVec;
  constexpr int UX = 1;
  const int t = threadIdx.x;
  if (t < h) fn(Elem<Tin>::load1(row, t));
  const vec4u* vp = reinterpret_cast<const vec4u*>(static_cast<const Tin*>(row) + h);
  vec4u v[LDX];
  stretch_prefetch<Tin, kTpBlock, LDX>(row, h, 0, nvec, v);
  stream_stretch<Tin, kTpBlock, UX, LDX>(vp, 0, nvec, v, [&](const vec4u* vv, int64_t) {
#pragma unroll
    for (int u = 0; u < UX; ++u) {
      float z[VEC];
      Elem<Tin>::unpack(vv[u], z);
#pragma unroll
      for (int k = 0; k < VEC; ++k) fn(z[k]);
    }
  });
  for (int64_t e = h + nvec * VEC + t; e < V; e += kTpBlock) fn(Elem<Tin>::load1(row, e));
}

// Block-wide sums of (x, y) in a fixed order; every thread gets the result.
__device__ __forceinline__ void block_sum2(double& x, double& y, TpShared& sh) {
  x = wave_sum_d(x);
  y = wave_sum_d(y);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if (threadIdx.x % kWave == 0) {
    sh.red_d[0][w] = x;
    sh.red_d[1][w] = y;
  }
  __syncthreads();
  x = 0.0;
  y = 0.0;
  for (int k = 0; k < kNW; ++k) {
    x += sh.red_d[0][k];
    y += sh.red_d[1][k];
  }
  __syncthreads();
}

__device__ __forceinline__ uint32_t block_sum_u(uint32_t v, TpShared& sh) {
  v = wave_sum_u(v);
  __syncthreads();
  if (threadIdx.x % kWave == 0) sh.red_u[threadIdx.x / kWave] = v;
  __syncthreads();
  uint32_t tot = 0;
  for (int k = 0; k < kNW; ++k) tot += sh.red_u[k];
  __syncthreads();
  return tot;
}

// Block-wide maxima of (a, b); every thread gets them.
__device__ __forceinline__ void block_max2_u(uint32_t& a, uint32_t& b, TpShared& sh) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) {
    a = max(a, static_cast<uint32_t>(__shfl_xor(static_cast<int>(a), o)));
    b = max(b, static_cast<uint32_t>(__shfl_xor(static_cast<int>(b), o)));
  }
  __syncthreads();
  if (threadIdx.x % kWave == 0) {
    sh.red_m[0][threadIdx.x / kWave] = a;
    sh.red_m[1][threadIdx.x / kWave] = b;
  }
  __syncthreads();
  a = 0u;
  b = 0u;
  for (int k = 0; k < kNW; ++k) {
    a = max(a, sh.red_m[0][k]);
    b = max(b, sh.red_m[1][k]);
  }
  __syncthreads();
}

// Exclusive block scan of one double per thread (thread order).
__device__ __forceinline__ double block_exclusive_scan(double v, TpShared& sh) {
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  double incl = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const double t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  __syncthreads();
  if (lane == kWave - 1) sh.red_d[0][w] = incl;
  __syncthreads();
  double base = 0.0;
  for (int k = 0; k < w; ++k) base += sh.red_d[0][k];
  __syncthreads();
  return base + incl - v;
}

struct Dist {
  float M;       // row maximum
  float invT;    // 1 / T (float32, for binning only)
  double invT64; // 1 / T
  __device__ __forceinline__ float nats(float z) const { return (M - z) * invT; }
  __device__ __forceinline__ int bin(float d) const {
    const int b = static_cast<int>(d * (kBins / kDMax));
    return b < kBins - 1 ? b : kBins - 1;
  }
  __device__ __forceinline__ double d64(float z) const {
    return (static_cast<double>(z) - static_cast<double>(M)) * invT64;
  }
};

// exp(d) for finite d in [-700, 0] (table-driven, Tang 1989): n = round(64 d
// / ln2) by adding and subtracting 1.5 * 2^52 (the low word of the sum is n),
// r = d - n ln2/64 in two parts (n * kLn2By64Hi is exact for |n| < 2^24),
// exp(r) by its degree-5 Taylor polynomial (|r| <= ln2/128: truncation below
// 4e-17), times 2^((n mod 64) / 64) from the table, times 2^(n div 64) built
// from its exponent bits.
__device__ __forceinline__ double exp_tang(double d, const double* tab) {
  constexpr double kInvLn2By64 = 0x1.71547652b82fep+6;  // 64 / ln2
  constexpr double kLn2By64Hi = 0x1.62e42fe000000p-7;
  constexpr double kLn2By64Lo = 0x1.f473de6af278fp-36;
  constexpr double kShift = 0x1.8p52;
  const double t = fma(d, kInvLn2By64, kShift);
  const int ni = static_cast<int>(static_cast<uint32_t>(__double_as_longlong(t)));
  const double n = t - kShift;
  double r = fma(-n, kLn2By64Hi, d);
  r = fma(-n, kLn2By64Lo, r);
  double p = fma(r, 1.0 / 120.0, 1.0 / 24.0);
  p = fma(p, r, 1.0 / 6.0);
  p = fma(p, r, 0.5);
  p = fma(p, r, 1.0);
  p = fma(p, r, 1.0);
  const double scale = __longlong_as_double(static_cast<long long>(static_cast<uint64_t>((ni >> 6) + 1023) << 52));
  return tab[ni & 63] * p * scale;
}

// Stats-pass histogram. A logit's bin coordinate is bf = (A0 - z) / T * kHK
// + kHAbove * kHK; it is formed scaled by kOffQ, x = fma(z, kz4, k04) with
// kz4 = kOffQ kz and k04 = kOffQ k0 (a power of two: x = kOffQ fma(z, kz, k0)
// exactly), so that one conversion gives the bin floor(bf) (the high bits of
// floor(x)) and the logit's position inside it (the low kOffBits bits:
// floor((bf - floor(bf)) kOffQ)). Both go to the bin in one 64-bit atomic;
// x < 0 (more than kHAbove nats above A0) goes to the list instead, bf >=
// kHB is beyond the window (no update). The exact pass recomputes x with
// the same operands, so both passes bin identically.
struct HistHook {
  uint64_t* bins;
  float* above;
  uint32_t* n_above;
  float kz, k0;    // bin coordinate bf = fma(z, kz, k0)
  float kz4, k04;  // the same scaled by kOffQ
  __device__ __forceinline__ void count(float z) {
    const float x = fmaf(z, kz4, k04);
    // Without a branch: the bits of x capped at those of kHB kOffQ (x is never
    // -0, since k04 is not; negative x, NaN and the infinities compare above
    // the cap) send every logit outside [0, kHB kOffQ) to bins[kHB].
    const uint32_t u = min(__float_as_uint(x), __float_as_uint(static_cast<float>(kHB) * kOffQ));
    const uint32_t xi = static_cast<uint32_t>(__uint_as_float(u));
    atomicAdd(&bins[xi >> kOffBits], (uint64_t{1} << kCountShift) | (xi & ((1u << kOffBits) - 1)));
  }
  template <int N>
  __device__ __forceinline__ void step(const float (&z)[N], const float (&)[N], float cmax, int64_t, const Lane&) {
#pragma unroll
    for (int k = 0; k < N; ++k) count(z[k]);
    if (__any(fmaf(cmax, kz4, k04) < 0.0f)) {  // x is non-increasing in z
#pragma unroll
      for (int k = 0; k < N; ++k) add_above(z[k]);
    }
  }
  __device__ __forceinline__ void scalar(float z, float, int64_t, const Lane&) {
    count(z);
    add_above(z);
  }
  __device__ __forceinline__ void finish(const Lane&) {}
  __device__ __forceinline__ void add_above(float z) {
    if (fmaf(z, kz4, k04) < 0.0f) {
      const uint32_t slot = atomicAdd(n_above, 1u);
      if (slot < static_cast<uint32_t>(kAboveCap)) above[slot] = z;
    }
  }
};

// Bitonic sort of sh.win[0..n2) into descending order (n2 a power of two).
__device__ __forceinline__ void bitonic_desc(float* a, int n2) {
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < (n2 >> 1); i += kTpBlock) {
        const int lo = 2 * stride * (i / stride) + (i % stride);
        const int hi = lo + stride;
        const bool desc = (lo & size) == 0;
        const float x = a[lo], y = a[hi];
        if (desc ? (x < y) : (x > y)) {
          a[lo] = y;
          a[hi] = x;
        }
      }
      __syncthreads();
    }
  }
}

// Radix refinement inside the crossing bins [b_lo, b_hi]: finds the boundary
// logit value and resolves ties by count. On entry sh.massAbove/Eabove/
// cntAbove hold the exact sums of the logits above b_lo. The digit masses
// are float atomics and only choose the digits; the masses that reach the
// result are summed again in a fixed order once the boundary value is known.
template <typename Tin>
__device__ Nucleus radix_boundary(const void* row, int32_t V, int64_t h, int64_t nvec, const Dist D, TpShared& sh) {
  const double massAbove0 = sh.massAbove, Eabove0 = sh.Eabove;
  const uint32_t blo = sh.b_lo, bhi = sh.b_hi;
  double massGT = massAbove0, EGT = Eabove0;
  uint32_t cntGT = sh.cntAbove;
  uint32_t prefix = 0, mask = 0, cnt_last = 0;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int b = threadIdx.x; b < 256; b += kTpBlock) {
      sh.r.rx.mass[b] = 0.0;
      sh.r.rx.E[b] = 0.0;
      sh.r.rx.cnt[b] = 0;
    }
    __syncthreads();
    for_each_logit<Tin>(row, V, h, nvec, [&](float z) {
      const float d = D.nats(z);
      if (!(d < kDMax)) return;
      const uint32_t b = static_cast<uint32_t>(D.bin(d));
      if (b < blo || b > bhi) return;
      const uint32_t key = float_key(z);
      if ((key & mask) != prefix) return;
      const uint32_t dg = (key >> shift) & 255u;
      const double dd = D.d64(z);
      const double e = exp(dd);
      atomicAdd(&sh.r.rx.mass[dg], e);
      atomicAdd(&sh.r.rx.E[dg], e * dd);
      atomicAdd(&sh.r.rx.cnt[dg], 1u);
    });
    __syncthreads();
    if (threadIdx.x == 0) {
      int dg = 255;
      for (; dg > 0; --dg) {  // descending keys: larger logits first
        if (massGT + sh.r.rx.mass[dg] >= sh.target) break;
        massGT += sh.r.rx.mass[dg];
        EGT += sh.r.rx.E[dg];
        cntGT += sh.r.rx.cnt[dg];
      }
      sh.rdigit = static_cast<uint32_t>(dg);
      sh.massAbove = massGT;
      sh.Eabove = EGT;
      sh.cntAbove = cntGT;
      sh.rcount = sh.r.rx.cnt[dg];
    }
    __syncthreads();
    prefix |= sh.rdigit << shift;
    mask |= 255u << shift;
    massGT = sh.massAbove;
    EGT = sh.Eabove;
    cntGT = sh.cntAbove;
    cnt_last = sh.rcount;
    __syncthreads();
  }
  // Exact sums over the crossing bins' logits above z* (larger keys), each
  // lane in its own fixed order, then a fixed-order block sum.
  {
    double gm = 0.0, ge = 0.0;
    for_each_logit<Tin>(row, V, h, nvec, [&](float z) {
      const float d = D.nats(z);
      if (!(d < kDMax)) return;
      const uint32_t b = static_cast<uint32_t>(D.bin(d));
      if (b < blo || b > bhi || float_key(z) <= prefix) return;
      const double dd = D.d64(z);
      const double e = exp(dd);
      gm += e;
      ge += e * dd;
    });
    block_sum2(gm, ge, sh);
    massGT = massAbove0 + gm;
    EGT = Eabove0 + ge;
  }
  // All remaining candidates share the value z*: equal masses e*.
  const float zs = key_float(prefix);
  const double dd = D.d64(zs);
  const double es = exp(dd);
  double jd = ceil((sh.target - massGT) / es);
  if (jd < 1.0) jd = 1.0;
  if (jd > static_cast<double>(cnt_last)) jd = static_cast<double>(cnt_last);
  const uint32_t j = static_cast<uint32_t>(jd);
  Nucleus n;
  n.k = static_cast<int32_t>(cntGT + j);
  n.S = massGT + static_cast<double>(j) * es;
  n.E = EGT + static_cast<double>(j) * es * dd;
  return n;
}

// The nucleus by the three-pass method (float64 histogram relative to M,
// exact sums above the crossing bins with their logits gathered, sorted and
// scanned; radix refinement when the crossing bins are overfull).
template <typename Tin>
__device__ Nucleus legacy_nucleus(const void* row, int32_t V, int64_t h, int64_t nvec, const Dist D, float P,
                                  TpShared& sh) {
  // histogram of the candidates' masses over distance bins
  __syncthreads();
  for (int b = threadIdx.x; b < kBins; b += kTpBlock) {
    sh.u.lg.mass[b] = 0.0;
    sh.u.lg.cnt[b] = 0;
  }
  if (threadIdx.x == 0) sh.wcount = 0;
  __syncthreads();
  double s64 = 0.0, unused = 0.0;
  for_each_logit<Tin>(row, V, h, nvec, [&](float z) {
    const float d = D.nats(z);
    if (!(d < kDMax)) return;
    const double e = exp(D.d64(z));
    const int b = D.bin(d);
    atomicAdd(&sh.u.lg.mass[b], e);
    atomicAdd(&sh.u.lg.cnt[b], 1u);
    s64 += e;
  });
  block_sum2(s64, unused, sh);  // fixed-order total: deterministic
  const double target = static_cast<double>(P) * s64;
  const double tol = 1e-9 * s64;

  // crossing bins: the first bins whose cumulative mass reaches target -/+ tol
  constexpr int kPer = kBins / kTpBlock;
  const int b0 = threadIdx.x * kPer;
  double seg = 0.0;
  for (int k = 0; k < kPer; ++k) seg += sh.u.lg.mass[b0 + k];
  const double before = block_exclusive_scan(seg, sh);
  if (threadIdx.x == 0) {
    sh.S64 = s64;
    sh.target = target;
    sh.b_lo = kBins - 1;
    sh.b_hi = kBins - 1;
  }
  __syncthreads();
  {
    double c = before;
    bool lo_done = false, hi_done = false;
    for (int k = 0; k < kPer; ++k) {
      c += sh.u.lg.mass[b0 + k];
      if (!lo_done && c >= target - tol) {
        atomicMin(&sh.b_lo, static_cast<uint32_t>(b0 + k));
        lo_done = true;
      }
      if (!hi_done && c >= target + tol) {
        atomicMin(&sh.b_hi, static_cast<uint32_t>(b0 + k));
        hi_done = true;
      }
    }
  }
  __syncthreads();
  const uint32_t b_lo = sh.b_lo, b_hi = sh.b_hi;
  uint32_t above = 0, inwin = 0;
  for (int k = 0; k < kPer; ++k) {
    const uint32_t b = static_cast<uint32_t>(b0 + k);
    if (b < b_lo) above += sh.u.lg.cnt[b];
    else if (b <= b_hi) inwin += sh.u.lg.cnt[b];
  }
  above = block_sum_u(above, sh);
  inwin = block_sum_u(inwin, sh);

  // exact sums above the crossing bins; gather the crossing bins' logits
  double mA = 0.0, eA = 0.0;
  const bool gather = inwin <= static_cast<uint32_t>(kCap);
  for_each_logit<Tin>(row, V, h, nvec, [&](float z) {
    const float d = D.nats(z);
    if (!(d < kDMax)) return;
    const uint32_t b = static_cast<uint32_t>(D.bin(d));
    if (b < b_lo) {
      const double dd = D.d64(z);
      const double e = exp(dd);
      mA += e;
      eA += e * dd;
    } else if (gather && b <= b_hi) {
      const uint32_t slot = atomicAdd(&sh.wcount, 1u);
      if (slot < static_cast<uint32_t>(kCap)) sh.win[slot] = z;
    }
  });
  block_sum2(mA, eA, sh);
  if (threadIdx.x == 0) {
    sh.massAbove = mA;
    sh.Eabove = eA;
    sh.cntAbove = above;
  }
  __syncthreads();

  Nucleus nuc;
  if (gather) {
    // sort the crossing logits (descending) and scan their masses
    const int nw = static_cast<int>(sh.wcount < static_cast<uint32_t>(kCap) ? sh.wcount : kCap);
    int n2 = 2;
    while (n2 < nw) n2 <<= 1;
    for (int i = nw + threadIdx.x; i < n2; i += kTpBlock) sh.win[i] = -INFINITY;
    __syncthreads();
    bitonic_desc(sh.win, n2);
    const int per = (n2 + kTpBlock - 1) / kTpBlock;
    const int i0 = threadIdx.x * per;
    const int i1 = i0 + per < nw ? i0 + per : nw;
    double sm = 0.0, se = 0.0;
    for (int i = i0; i < i1; ++i) {
      const double dd = D.d64(sh.win[i]);
      const double e = exp(dd);
      sm += e;
      se += e * dd;
    }
    const double cm = block_exclusive_scan(sm, sh);
    const double ce = block_exclusive_scan(se, sh);
    if (threadIdx.x == 0) sh.jfirst = 0xffffffffu;
    __syncthreads();
    // The running mass increases along the sorted logits: the first index
    // whose running mass reaches the target is the smallest one reported.
    double run_m = mA + cm;
    for (int i = i0; i < i1; ++i) {
      run_m += exp(D.d64(sh.win[i]));
      if (run_m >= target) {
        atomicMin(&sh.jfirst, static_cast<uint32_t>(i));
        break;
      }
    }
    __syncthreads();
    const uint32_t jf = sh.jfirst;
    if (jf != 0xffffffffu && static_cast<int>(jf) >= i0 && static_cast<int>(jf) < i1) {
      double m2 = mA + cm, e2 = eA + ce;
      for (int i = i0; i <= static_cast<int>(jf); ++i) {
        const double dd = D.d64(sh.win[i]);
        const double e = exp(dd);
        m2 += e;
        e2 += e * dd;
      }
      sh.SN = m2;
      sh.EN = e2;
    }
    __syncthreads();
    if (jf == 0xffffffffu) {
      // Not reached inside the gathered logits (only through rounding at
      // the very end of the order): the nucleus is everything gathered.
      double tm = sm, te = se;
      block_sum2(tm, te, sh);
      nuc.k = static_cast<int32_t>(above + static_cast<uint32_t>(nw));
      nuc.S = mA + tm;
      nuc.E = eA + te;
    } else {
      nuc.k = static_cast<int32_t>(above + jf + 1);
      nuc.S = sh.SN;
      nuc.E = sh.EN;
    }
  } else {
    nuc = radix_boundary<Tin>(row, V, h, nvec, D, sh);
  }
  return nuc;
}

// Lanes of a workgroup that may re-read their whole stretch in the sparse
// exact pass (a lane with three or more buckets reaching the window); with
// more, the row takes the dense pass.
constexpr uint32_t kSparseFullLanes = 16;
// Bound on the relative error of a bin's mass as estimated from its count
// and offset sum (first order around the centre), per logit: the second-order
// term (|x| <= 0.5 bin + 2.5e-4 bin of float32 rounding of the coordinate,
// at 0.0183 nats per bin) is below 4.24e-5 of the centre's mass, the
// quantised offsets and the coordinate's rounding add 6.7e-6; 5.5e-5 keeps a
// margin (the exact map from the float32 coordinate to nats is used).
constexpr double kBinMassRelErr = 5.5e-5;

// The window of bins around P of the total, located from the histogram.
struct Window {
  int b_lo, b_hi;       // bins of the window (-1: the list above the bins)
  uint32_t above;       // logits above the window (exact, from the counts and the list)
  uint32_t inwin;       // logits in the window (exact)
  double s_below;       // estimated mass of the bins below the window (relative to M)
  double s_below_err;   // bound on the error of s_below
};

// Calls fn(z) for the logits of the row that the sparse exact pass reads:
// every scalar head/tail logit, the lane's whole stretch when `full`, else
// the buckets (U = 2 vectors each) starting at vector indices s1 and s2
// (-1: none). Unread vectors cannot hold a logit at or above the window.
template <typename Tin, typename Fn>
__device__ __forceinline__ void for_each_listed_logit(const void* row, int32_t V, int64_t h, int64_t nvec, bool full,
                                                      int64_t s1, int64_t s2, Fn fn) {
  constexpr int VEC = Elem<Tin>::kVec;
  const int t = threadIdx.x;
  if (t < h) fn(Elem<Tin>::load1(row, t));
  for (int64_t e = h + nvec * VEC + t; e < V; e += kTpBlock) fn(Elem<Tin>::load1(row, e));
  const vec4u* vp = reinterpret_cast<const vec4u*>(static_cast<const Tin*>(row) + h);
  auto body = [&](const vec4u& x) {
    float z[VEC];
    Elem<Tin>::unpack(x, z);
#pragma unroll
    for (int k = 0; k < VEC; ++k) fn(z[k]);
  };
  if (full) {
    int64_t v = t;
    for (; v + kTpBlock < nvec; v += 2 * kTpBlock) {
      const vec4u x0 = load_stream(vp + v);
      const vec4u x1 = load_stream(vp + v + kTpBlock);
      body(x0);
      body(x1);
    }
    if (v < nvec) body(load_stream(vp + v));
    return;
  }
  const int64_t idx[4] = {s1, s1 + kTpBlock, s2, s2 + kTpBlock};
  vec4u x[4];
  bool ok[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    ok[u] = (u < 2 ? s1 : s2) >= 0 && idx[u] < nvec;
    x[u] = ok[u] ? load_stream(vp + idx[u]) : neg_inf_vec<Tin>();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
    if (ok[u]) body(x[u]);
}

// Inclusive prefix sum over the lanes of a wave, in a fixed order.
__device__ __forceinline__ double wave_incl_scan_d(double x) {
  const int lane = static_cast<int>(threadIdx.x % kWave);
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const double t = __shfl_up(x, d);
    if (lane >= d) x += t;
  }
  return x;
}

// Sorts the 64 E floats a wave holds, E per lane (element E lane + k), into
// descending order with the same bitonic network as bitonic_desc: strides
// below E compare registers of one lane, longer ones the same register of
// lane ^ (stride / E).
template <int E>
__device__ __forceinline__ void wave_bitonic_desc(float (&v)[E]) {
  const int lane = static_cast<int>(threadIdx.x % kWave);
#pragma unroll
  for (int size = 2; size <= kWave * E; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= E) {
#pragma unroll
        for (int k = 0; k < E; ++k) {
          const int i = E * lane + k;
          const float p = __shfl_xor(v[k], stride / E);
          const bool keep_max = ((i & size) == 0) == ((i & stride) == 0);
          v[k] = keep_max ? fmaxf(v[k], p) : fminf(v[k], p);
        }
      } else {
#pragma unroll
        for (int k = 0; k < E; ++k) {
          if (k & stride) continue;
          const bool desc = ((E * lane + k) & size) == 0;
          const float a = v[k], b = v[k | stride];
          v[k] = desc ? fmaxf(a, b) : fminf(a, b);
          v[k | stride] = desc ? fminf(a, b) : fmaxf(a, b);
        }
      }
    }
  }
}

// cut_window for a window of at most 64 E logits: wave 0 holds it in
// registers, E per lane, sorts it, forms each mass once and scans with wave
// prefix sums (no workgroup barrier until the result is published). Same
// result as the workgroup-wide version up to the order of float64 additions.
template <int E, typename DD, typename Thr>
__device__ __forceinline__ bool cut_window_wave(TpShared& sh, int nw, uint32_t cA, double mA, double eA, DD dd_of,
                                                Thr thr, Nucleus& nuc) {
  const double* tab = sh.exptab;
  if (threadIdx.x < kWave) {
    const int lane = static_cast<int>(threadIdx.x);
    float v[E];
#pragma unroll
    for (int k = 0; k < E; ++k) v[k] = E * lane + k < nw ? sh.win[E * lane + k] : -INFINITY;
    wave_bitonic_desc<E>(v);
    double e[E], ed[E];
    double ls = 0.0, le = 0.0;
#pragma unroll
    for (int k = 0; k < E; ++k) {
      e[k] = 0.0;
      ed[k] = 0.0;
      if (E * lane + k < nw) {  // the window's logits lead the sorted order (the padding is -inf)
        const double dd = dd_of(v[k]);
        e[k] = exp_tang(dd, tab);
        ed[k] = e[k] * dd;
      }
      ls += e[k];
      le += ed[k];
    }
    const double is = wave_incl_scan_d(ls), ie = wave_incl_scan_d(le);
    // sums over the lanes before this one (the shuffles run in every lane: a
    // shuffle must not read a lane that is not executing it)
    const double pis = __shfl_up(is, 1), pie = __shfl_up(ie, 1);
    const double cm = lane > 0 ? pis : 0.0;
    const double ce = lane > 0 ? pie : 0.0;
    const double wm = __shfl(is, kWave - 1);
    double t_lo, t_hi;
    thr(wm, t_lo, t_hi);
    constexpr int kNone = 1 << 30;
    int jlo = kNone, jhi = kNone;
    const bool inside = mA < t_lo && !(mA + wm < t_hi);  // else the crossing lies outside the window
    if (inside) {
      double run = mA + cm;
#pragma unroll
      for (int k = 0; k < E; ++k) {
        run += e[k];
        if (jlo == kNone && run >= t_lo) jlo = E * lane + k;
        if (jhi == kNone && run >= t_hi) jhi = E * lane + k;
      }
    }
    // indices grow with the lane: the first lane that has one holds the smallest
    const uint64_t mlo = __ballot(jlo != kNone), mhi = __ballot(jhi != kNone);
    const int jf = mlo ? __shfl(jlo, static_cast<int>(__builtin_ctzll(mlo))) : kNone;
    const int jr = mhi ? __shfl(jhi, static_cast<int>(__builtin_ctzll(mhi))) : kNone;
    const bool decided = inside && jf != kNone && jf == jr;
    if (decided && jf / E == lane) {
      double m2 = mA + cm, e2 = eA + ce;
#pragma unroll
      for (int k = 0; k < E; ++k) {
        if (k <= jf % E) {
          m2 += e[k];
          e2 += ed[k];
        }
      }
      sh.SN = m2;
      sh.EN = e2;
    }
    if (lane == 0) sh.jfirst = decided ? static_cast<uint32_t>(jf) : 0xffffffffu;
  }
  __syncthreads();
  const uint32_t jf = sh.jfirst;
  if (jf == 0xffffffffu) return false;
  nuc.k = static_cast<int32_t>(cA + jf + 1);
  nuc.S = sh.SN;
  nuc.E = sh.EN;
  return true;
}

// cut_window for a window of at most 512 logits: the one-wave cut with the
// fewest logits per lane that holds it.
template <typename DD, typename Thr>
__device__ __forceinline__ bool cut_window_small(TpShared& sh, int nw, uint32_t cA, double mA, double eA, DD dd_of,
                                                 Thr thr, Nucleus& nuc) {
  if (nw <= kWave) return cut_window_wave<1>(sh, nw, cA, mA, eA, dd_of, thr, nuc);
  if (nw <= 2 * kWave) return cut_window_wave<2>(sh, nw, cA, mA, eA, dd_of, thr, nuc);
  if (nw <= 4 * kWave) return cut_window_wave<4>(sh, nw, cA, mA, eA, dd_of, thr, nuc);
  return cut_window_wave<8>(sh, nw, cA, mA, eA, dd_of, thr, nuc);
}

// cut_window for any window of at most kCap logits: a workgroup-wide
// bitonic sort, then block scans.
template <typename DD, typename Thr>
__device__ bool cut_window_block(TpShared& sh, int nw, uint32_t cA, double mA, double eA, DD dd_of, Thr thr,
                                 Nucleus& nuc) {
  const double* tab = sh.exptab;
  int n2 = 2;
  while (n2 < nw) n2 <<= 1;
  for (int i = nw + threadIdx.x; i < n2; i += kTpBlock) sh.win[i] = -INFINITY;
  __syncthreads();
  bitonic_desc(sh.win, n2);
  const int per = (n2 + kTpBlock - 1) / kTpBlock;
  const int i0 = threadIdx.x * per;
  const int i1 = i0 + per < nw ? i0 + per : nw;
  double sm = 0.0, se = 0.0;
  for (int i = i0; i < i1; ++i) {
    const double dd = dd_of(sh.win[i]);
    const double e = exp_tang(dd, tab);
    sm += e;
    se += e * dd;
  }
  const double cm = block_exclusive_scan(sm, sh);
  const double ce = block_exclusive_scan(se, sh);
  double wm = sm, we = se;
  block_sum2(wm, we, sh);
  double t_lo, t_hi;
  thr(wm, t_lo, t_hi);
  if (!(mA < t_lo) || mA + wm < t_hi) return false;  // crossing outside the window
  if (threadIdx.x == 0) {
    sh.jfirst = 0xffffffffu;
    sh.rdigit = 0xffffffffu;  // the first index reaching t_hi
  }
  __syncthreads();
  double run_m = mA + cm;
  bool lo_found = false;
  for (int i = i0; i < i1; ++i) {
    run_m += exp_tang(dd_of(sh.win[i]), tab);
    if (!lo_found && run_m >= t_lo) {
      atomicMin(&sh.jfirst, static_cast<uint32_t>(i));
      lo_found = true;
    }
    if (run_m >= t_hi) {
      atomicMin(&sh.rdigit, static_cast<uint32_t>(i));
      break;
    }
  }
  __syncthreads();
  const uint32_t jf = sh.jfirst;
  if (jf == 0xffffffffu || jf != sh.rdigit) return false;  // not decided within the bound
  if (static_cast<int>(jf) >= i0 && static_cast<int>(jf) < i1) {
    double m2 = mA + cm, e2 = eA + ce;
    for (int i = i0; i <= static_cast<int>(jf); ++i) {
      const double dd = dd_of(sh.win[i]);
      const double e = exp_tang(dd, tab);
      m2 += e;
      e2 += e * dd;
    }
    sh.SN = m2;
    sh.EN = e2;
  }
  __syncthreads();
  nuc.k = static_cast<int32_t>(cA + jf + 1);
  nuc.S = sh.SN;
  nuc.E = sh.EN;
  return true;
}

__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// cut_window for a window of more than 512 logits. Its logits fall into kSub
// sub-buckets by their order-preserving keys (sub-bucket 0 holds the largest
// values; equal values share one), and each sub-bucket sums its count, masses
// and entropy terms in 64-bit fixed point with integer atomics, so that the
// sums do not depend on the order of the additions. The sub-buckets before
// the first one whose running mass can reach the target lie above the cutoff
// whole; the logits of the sub-buckets in which the crossing can fall move to
// the front of sh.win and are cut alone, from the mass, entropy sum and count
// above them. A fixed-point mass errs by less than one unit (mref 2^-48), so
// the target interval is widened by twice the error of those sums: a cutoff
// taken inside the wider interval is the cutoff of the narrower one.
template <typename DD, typename Thr>
__device__ __forceinline__ bool cut_window_sub(TpShared& sh, int nw, uint32_t cA, double mA, double eA, DD dd_of,
                                               Thr thr, Nucleus& nuc) {
  constexpr int kPer = kCap / kTpBlock;
  constexpr uint32_t kNone = 0xffffffffu;
  const double* tab = sh.exptab;
  float z[kPer];
  uint32_t key[kPer];
  uint32_t kmax = 0u, knmin = 0u;  // largest key, largest complemented key
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int i = static_cast<int>(threadIdx.x) + k * kTpBlock;
    z[k] = i < nw ? sh.win[i] : 0.0f;
    key[k] = float_key(z[k]);
    if (i < nw) {
      kmax = max(kmax, key[k]);
      knmin = max(knmin, ~key[k]);
    }
  }
  if (threadIdx.x < kSub) {
    sh.r.sb.q[threadIdx.x] = 0ull;
    sh.r.sb.qe[threadIdx.x] = 0ull;
    sh.r.sb.cnt[threadIdx.x] = 0u;
  }
  block_max2_u(kmax, knmin, sh);  // its barriers also order the clearing before the sums
  const uint32_t hi = kmax, span = kmax - ~knmin;
  const int shift = span < static_cast<uint32_t>(kSub) ? 0 : 24 - __builtin_clz(span);  // span >> shift < kSub
  const double dd_hi = dd_of(key_float(hi)), dd_lo = dd_of(key_float(~knmin));
  const double mref = exp_tang(dd_hi, tab) * (1.0 + 0x1p-30);  // at least every mass of the window
  if (!(mref > 0x1p-900 && mref < 0x1p900)) return cut_window_block(sh, nw, cA, mA, eA, dd_of, thr, nuc);
  const double scale = 0x1p48 / mref;
  const double scale_e = 0x1p48 / (mref * fmax(fmax(fabs(dd_hi), fabs(dd_lo)), 1.0));
  int sb[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int i = static_cast<int>(threadIdx.x) + k * kTpBlock;
    sb[k] = static_cast<int>((hi - key[k]) >> shift);
    if (i < nw) {
      const double dd = dd_of(z[k]);
      const double e = exp_tang(dd, tab);
      atomicAdd(&sh.r.sb.q[sb[k]], static_cast<unsigned long long>(e * scale));
      atomicAdd(&sh.r.sb.qe[sb[k]], static_cast<unsigned long long>(static_cast<long long>(e * dd * scale_e)));
      atomicAdd(&sh.r.sb.cnt[sb[k]], 1u);
    }
  }
  __syncthreads();
  if (threadIdx.x < kWave) {
    // wave 0: kSub / 64 consecutive sub-buckets per lane, scanned in order
    constexpr int kPL = kSub / kWave;
    const int lane = static_cast<int>(threadIdx.x);
    double m[kPL], ee[kPL], c[kPL];
    double lm = 0.0, le = 0.0, lc = 0.0;
#pragma unroll
    for (int j = 0; j < kPL; ++j) {
      const int s = kPL * lane + j;
      m[j] = static_cast<double>(sh.r.sb.q[s]) / scale;
      ee[j] = static_cast<double>(static_cast<long long>(sh.r.sb.qe[s])) / scale_e;
      c[j] = static_cast<double>(sh.r.sb.cnt[s]);
      lm += m[j];
      le += ee[j];
      lc += c[j];
    }
    const double ism = wave_incl_scan_d(lm), ise = wave_incl_scan_d(le), isc = wave_incl_scan_d(lc);
    const double pm = __shfl_up(ism, 1), pe = __shfl_up(ise, 1), pc = __shfl_up(isc, 1);
    const double wm = __shfl(ism, kWave - 1);
    double t_lo, t_hi;
    thr(wm, t_lo, t_hi);
    // each fixed-point mass is low by less than 1 / scale; the conversions and
    // the float64 sums add a few units in the last place
    const double err = (static_cast<double>(nw) + 8.0) / scale + 1e-14 * (fabs(mA) + wm);
    t_lo -= 2.0 * err;
    t_hi += 2.0 * err;
    const bool inside = mA < t_lo && !(mA + wm < t_hi);
    int slo = kSub, shi = kSub;
    double run = mA + (lane > 0 ? pm : 0.0);
#pragma unroll
    for (int j = 0; j < kPL; ++j) {
      run += m[j];
      if (slo == kSub && run >= t_lo) slo = kPL * lane + j;
      if (shi == kSub && run >= t_hi) shi = kPL * lane + j;
    }
    const uint64_t mlo = __ballot(slo < kSub), mhi = __ballot(shi < kSub);
    const int sf = mlo ? __shfl(slo, static_cast<int>(__builtin_ctzll(mlo))) : kSub;
    const int sl = mhi ? __shfl(shi, static_cast<int>(__builtin_ctzll(mhi))) : kSub;
    const bool ok = inside && sf < kSub && sl < kSub;
    if (ok && sf / kPL == lane) {  // the sums over the sub-buckets before sf
      double bm = mA + (lane > 0 ? pm : 0.0), be = eA + (lane > 0 ? pe : 0.0), bc = lane > 0 ? pc : 0.0;
#pragma unroll
      for (int j = 0; j < kPL; ++j) {
        if (j < sf % kPL) {
          bm += m[j];
          be += ee[j];
          bc += c[j];
        }
      }
      sh.sc.m = bm;
      sh.sc.e = be;
      sh.sc.c = cA + static_cast<uint32_t>(bc);
    }
    if (lane == 0) {
      sh.sc.t_lo = t_lo;
      sh.sc.t_hi = t_hi;
      sh.sc.s_first = ok ? static_cast<uint32_t>(sf) : kNone;
      sh.sc.s_last = static_cast<uint32_t>(sl);
      sh.wcount = 0u;
    }
  }
  __syncthreads();
  const uint32_t sf = sh.sc.s_first, sl = sh.sc.s_last;
  if (sf == kNone) return false;
  // every thread holds its logits in registers: the window can be rewritten
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int i = static_cast<int>(threadIdx.x) + k * kTpBlock;
    if (i < nw && static_cast<uint32_t>(sb[k]) >= sf && static_cast<uint32_t>(sb[k]) <= sl) {
      const uint32_t slot = atomicAdd(&sh.wcount, 1u);
      sh.win[slot] = z[k];
    }
  }
  __syncthreads();
  const int nc = static_cast<int>(sh.wcount);
  const double t_lo = sh.sc.t_lo, t_hi = sh.sc.t_hi, bm = sh.sc.m, be = sh.sc.e;
  const uint32_t bc = sh.sc.c;
  auto thr_c = [&](double, double& lo, double& hi_) {
    lo = t_lo;
    hi_ = t_hi;
  };
  if (nc <= 512) return cut_window_small(sh, nc, bc, bm, be, dd_of, thr_c, nuc);
  return cut_window_block(sh, nc, bc, bm, be, dd_of, thr_c, nuc);
}

// Step 3 of the histogram method: the window's nw_all logits (in sh.win)
// sorted into descending order and scanned. A logit's mass is exp(dd(z)) in
// the caller's frame; mA and eA are the mass and the entropy sum (nats of
// that frame) above the window, cA the number of logits there. The cutoff
// is the first index j at which the running mass mA + C_j reaches the
// target; thr(wm, t_lo, t_hi) gives the interval [t_lo, t_hi] the target
// may lie in (wm: the window's total mass), and j is taken only where both
// ends give the same index. Returns false when they do not, or when the
// crossing lies outside the window; else the nucleus size and its mass and
// entropy sums in the caller's frame.
template <typename DD, typename Thr>
__device__ bool cut_window(TpShared& sh, uint32_t nw_all, uint32_t cA, double mA, double eA, DD dd_of, Thr thr,
                           Nucleus& nuc) {
  const int nw = static_cast<int>(nw_all);
  if (nw <= 512) return cut_window_small(sh, nw, cA, mA, eA, dd_of, thr, nuc);
  return cut_window_sub(sh, nw, cA, mA, eA, dd_of, thr, nuc);
}

// Steps 2 and 3 of the histogram method: the exact pass over the row (dense)
// or over the buckets that can reach the window (sparse), the window sorted
// and scanned. Dense: S is the float64 total over every binned logit.
// Sparse: S is the exact mass at or above the window plus the histogram's
// estimate of the mass below it, whose error is bounded; the cutoff is taken
// only where the whole uncertainty interval of P * S leads to the same index,
// and the logits read must account for every counted logit at or above the
// window. Returns false when the method cannot decide (the caller then tries
// the dense pass, then the three-pass method).
template <typename Tin, bool SPARSE>
__device__ __forceinline__ bool exact_cut(const void* row, int32_t V, int64_t h, int64_t nvec, const Dist& D, float P,
                          const HistHook& hk, TpShared& sh, const Window& W, double c0, double invK, bool full,
                          int64_t s1, int64_t s2, Nucleus& nuc) {
  const double* tab = sh.exptab;
  const int b_lo = W.b_lo, b_hi = W.b_hi;
  if (threadIdx.x == 0) sh.wcount = 0;
  __syncthreads();
  // 2. exact pass: sums above the window, the window gathered, the total
  // (every binned logit: those more than 50 nats below M add less than
  // V e^-50 of S). With u = (z - M) / T - c0 by one fma (the row constant
  // -M / T - c0 is rounded once: a common factor of every mass, which the
  // cutoff test does not see), a logit of bin b sits r = u + b / kHK from
  // its bin centre and dd = u + c0 nats below M; the entropy sum above the
  // window is taken as sum e u + c0 * sum e.
  double mA = 0.0, eAu = 0.0, sT = 0.0;
  uint32_t nA = 0;
  const double nMTc = -static_cast<double>(D.M) * D.invT64 - c0;
  auto visit = [&](float z) {
    const float x = fmaf(z, hk.kz4, hk.k04);
    if (!(x < static_cast<float>(kHB) * kOffQ)) return;  // beyond 50 nats below A0, -inf, NaN
    const double u = fma(static_cast<double>(z), D.invT64, nMTc);
    double e;
    int b;
    if (x >= 0.0f) {
      b = static_cast<int>(static_cast<uint32_t>(x) >> kOffBits);
      if (SPARSE && b > b_hi) return;  // below the window: estimated from the histogram
      const double r = fma(static_cast<double>(b), invK, u);
      const float rf = static_cast<float>(r);
      const float cf = fmaf(rf, fmaf(rf, 1.0f / 120.0f, 1.0f / 24.0f), 1.0f / 6.0f);
      double q = fma(static_cast<double>(cf), r, 0.5);
      q = fma(q, r, 1.0);
      q = fma(q, r, 1.0);
      e = sh.u.wtab[b] * q;
    } else {
      b = -1;  // the list above the bins
      e = exp_tang(fmax(u + c0, -700.0), tab);
    }
    if (!SPARSE) sT += e;
    if (b < b_lo) {  // above the window (lanes outside it keep their sums as they are)
      mA += e;
      eAu = fma(e, u, eAu);
      if (SPARSE) ++nA;
    } else if (b <= b_hi) {
      const uint32_t slot = atomicAdd(&sh.wcount, 1u);
      if (slot < static_cast<uint32_t>(kCap)) sh.win[slot] = z;
    }
  };
  if (SPARSE)
    for_each_listed_logit<Tin>(row, V, h, nvec, full, s1, s2, visit);
  else
    for_each_logit<Tin>(row, V, h, nvec, visit);
  block_sum2(mA, eAu, sh);
  const double eA = fma(c0, mA, eAu);
  double sT2 = sT, unused = 0.0;
  if (!SPARSE) block_sum2(sT2, unused, sh);
  const uint32_t cA = W.above;
  const uint32_t nw_all = sh.wcount;
  if (nw_all > static_cast<uint32_t>(kCap)) return false;
  if (SPARSE) {  // every counted logit at or above the window was read
    const uint32_t nA_all = block_sum_u(nA, sh);
    if (nA_all != cA || nw_all != W.inwin) return false;
  }

  return cut_window(
      sh, nw_all, cA, mA, eA, [&](float z) { return D.d64(z); },
      [&](double wm, double& t_lo, double& t_hi) {
        // The total and the range the target P * S may lie in: exact (to
        // float64 rounding) in the dense pass, the histogram estimate's bound
        // in the sparse one.
        const double S = SPARSE ? mA + wm + W.s_below : sT2;
        const double err = SPARSE ? W.s_below_err + 1e-13 * S : 0.0;
        t_lo = static_cast<double>(P) * (S - err);
        t_hi = static_cast<double>(P) * (S + err);
      },
      nuc);
}

// Step 2 in float32, for rows whose window many buckets reach (the flat
// ones). One pass forms every binned logit's mass as 2^t, t = z c + nMc with
// c = log2(e) / T held as a float pair (two fmas) and nMc = -M c + shift
// rounded to float (the frame: every mass carries the common factor 2^tau,
// tau = nMc + M c; the shift puts t = 0 at the window), by the hardware
// exp2; float64 sums of the masses and of m t over every binned logit and
// over those above the window; the window gathered. The window's masses are then taken exactly (float64) in
// the same frame, and the cutoff only where the certified error of the
// float32 masses leaves one index. The bound: a logit's t errs by at most
// 2^-23 |t| + 2^-47 max|z| c (two roundings of |t| and the float pair's
// remainder), so its mass by ln2 (2^-23 |t| + 2^-47 max|z| c) + kExp2RelErr
// relative (for t >= -100; below, at most 2^-100 absolute). With mass
// errors d_A above the window and d_R in the rest (window included, since
// the total is the float32 sum), the test quantity mA + C_j - P S errs by at
// most (1 - P) d_A + P d_R. Returns false when that does not decide (the
// caller then takes the float64 pass); else the nucleus relative to M.
template <typename Tin>
__device__ __forceinline__ bool approx_cut(const void* row, int32_t V, int64_t h, int64_t nvec, const Dist& D, float P, float A0,
                           const HistHook& hk, TpShared& sh, const Window& W, Nucleus& nuc) {
  if (threadIdx.x == 0) sh.wcount = 0;
  __syncthreads();
  const double c64 = kLog2eD * D.invT64;
  const float c_hi = static_cast<float>(c64);
  const float c_lo = static_cast<float>(c64 - static_cast<double>(c_hi));
  // The frame puts t = 0 near the window (bin b_lo's centre, at most 100
  // above M's t): the rounding error of t grows with |t|, and the logits
  // that decide the cutoff are the massive ones and those near the window.
  const double zw = W.b_lo >= 0 ? (static_cast<double>(W.b_lo) + 0.5 - static_cast<double>(hk.k0)) /
                                      static_cast<double>(hk.kz)
                                : static_cast<double>(D.M);
  const double shift = fmin((static_cast<double>(D.M) - zw) * c64, 100.0);
  const float nMc = static_cast<float>(-static_cast<double>(D.M) * c64 + fmax(shift, 0.0));
  const double nMc64 = static_cast<double>(nMc);
  const float xa = W.b_lo >= 0 ? static_cast<float>(W.b_lo) * kOffQ : -INFINITY;  // above the window: x < xa
  const float xb = static_cast<float>(W.b_hi + 1) * kOffQ;                       // in it: xa <= x < xb
  double sT = 0.0, tT = 0.0, mA = 0.0, tA = 0.0;
  auto visit = [&](float z) {
    const float x = fmaf(z, hk.kz4, hk.k04);
    if (!(x < static_cast<float>(kHB) * kOffQ)) return;  // the binned logits, as in the exact pass
    const float t = fmaf(z, c_lo, fmaf(z, c_hi, nMc));
    const float e = __builtin_amdgcn_exp2f(t);
    const double e64 = static_cast<double>(e);
    const double t64 = static_cast<double>(t);
    sT += e64;
    tT = fma(e64, t64, tT);  // the product is exact: one rounding either way
    if (x < xa) {
      mA += e64;
      tA = fma(e64, t64, tA);
    } else if (x < xb) {
      const uint32_t slot = atomicAdd(&sh.wcount, 1u);
      if (slot < static_cast<uint32_t>(kCap)) sh.win[slot] = z;
    }
  };
  for_each_logit<Tin, approx_depth<Tin>()>(row, V, h, nvec, visit);
  block_sum2(sT, tT, sh);
  block_sum2(mA, tA, sh);
  const uint32_t nw_all = sh.wcount;
  if (nw_all > static_cast<uint32_t>(kCap) || nw_all != W.inwin) return false;
  // the bound (sums of the float32 masses, inflated for their own error)
  const double T = 1.0 / D.invT64;
  const double zc = fmax(fabs(static_cast<double>(D.M)), fabs(static_cast<double>(A0)) + 50.0 * T) * c64;
  const double g1 = kLn2D * 0x1p-23 * 1.0001;                           // per unit of m |t|
  const double g0 = (kLn2D * 0x1p-47 * zc + kExp2RelErr) * 1.0001;     // per unit of m
  // sums of m |t|: in this frame a logit above the window has t > -kTSlack
  // and any other one t < kTSlack (half a bin is 0.0132 in t, plus the
  // roundings of the bin coordinate and of nMc)
  const double aA = tA + 2.0 * kTSlack * mA;                     // above the window
  const double aR = (tA - tT) + 2.0 * kTSlack * (sT - mA);       // the rest
  const double d_above = (g1 * aA + g0 * mA) * (1.0 + 1e-6);
  const double d_rest = (g1 * aR + g0 * (sT - mA)) * (1.0 + 1e-6);
  const double Pd = static_cast<double>(P);
  const double dF = (1.0 - Pd) * d_above + Pd * fmax(d_rest, 0.0) + static_cast<double>(V) * (0x1p-99 + 2e-22) +
                    1e-12 * sT;
  const double tau_n = kLn2D * (nMc64 + static_cast<double>(D.M) * c64);  // the frame's offset, in nats
  const bool ok = cut_window(
      sh, nw_all, W.above, mA, kLn2D * tA, [&](float z) { return kLn2D * fma(static_cast<double>(z), c64, nMc64); },
      [&](double, double& t_lo, double& t_hi) {
        t_lo = Pd * sT - dF;
        t_hi = Pd * sT + dF;
      },
      nuc);
  if (!ok) return false;
  // from the frame to masses relative to M: m_M = m / e^tau_n, d_M = d - tau_n
  const double inv_kappa = exp(-tau_n);
  nuc.E = (nuc.E - tau_n * nuc.S) * inv_kappa;
  nuc.S *= inv_kappa;
  return true;
}

// The nucleus from the stats-pass histogram and one exact pass (sparse when
// few buckets can reach the window, else dense). Returns false (and leaves
// nuc unset) when the row must take the three-pass method. tk holds each
// lane's three largest bucket maxima and the steps of the first two.
template <typename Tin>
__device__ __forceinline__ bool hist_nucleus(const void* row, int32_t V, int64_t h, int64_t nvec, const Dist& D, float P,
                             float A0, const HistHook& hk, const topk::Hook& tk, TpShared& sh, Nucleus& nuc) {
  const double* tab = sh.exptab;
  const uint32_t n_above = sh.n_above;
  if (n_above > static_cast<uint32_t>(kAboveCap)) return false;
  // The float32 bin coordinate bf is within a fraction of a bin of the exact
  // one while |k0| < 2^18 (kz and k0 carry a relative error below 2.4e-7,
  // and a binned logit has |z kz| < |k0| + kHB): every binned logit then
  // lies within 0.012 nats of its bin centre, where the exact pass's
  // degree-5 polynomial is accurate to 3e-14. Rows with larger |A0| / T
  // (beyond about 4,800) take the three-pass method.
  if (!(fabsf(hk.k0) < 0x1p18f)) return false;

  // 1. the window of bins around P * (total). bf = z kz + k0 (the float32
  // constants, exactly) is a logit's coordinate: it lies (M - z) / T =
  // bf * hb - lead nats below M, with hb = -1 / (kz T) and lead = -(M + k0 /
  // kz) / T, so that the only error of the rounded coordinate is its last
  // rounding. A bin's mass is taken at its centre, corrected to first order
  // by the offsets: w_b (count - hb * sum of offsets) with w_b the mass at
  // the centre (relative error below kBinMassRelErr per logit).
  const double hb = -D.invT64 / static_cast<double>(hk.kz);
  const double lead = -(static_cast<double>(D.M) + static_cast<double>(hk.k0) / static_cast<double>(hk.kz)) * D.invT64;
  const double invK = 1.0 / static_cast<double>(kHK);
  // Kept compact (it runs once per row): the loops over a thread's kPer bins
  // are not unrolled (one copy of the float64 exp each; the second loop
  // recomputes the masses of the first), and the crossing bins are found
  // with a ballot and one LDS atomic per wave.
  // A thread's kPer consecutive bins: centre masses by the recurrence
  // w_{b+1} = w_b * exp(-hb) from one exp per thread (kPer - 1 roundings,
  // below 1e-15 relative).
  constexpr int kPer = kHB / kTpBlock;
  const int b0 = threadIdx.x * kPer;
  const double w0 = exp(fma(-(static_cast<double>(b0) + 0.5), hb, lead));
  const double rho = exp(-hb);
  auto bin_mass = [&](int b, double w) -> double {
    const uint64_t word = sh.u.hs.bins[b];
    const double cnt = static_cast<double>(static_cast<uint32_t>(word >> kCountShift));
    // a position p stands for the offset (p + 1/2) / kOffQ - 1/2 from the centre
    const double dsum =
        (static_cast<double>(word & ((uint64_t{1} << kCountShift) - 1)) - cnt * (0.5 * kOffQ - 0.5)) * (1.0 / kOffQ);
    return fma(-dsum, hb, cnt) * w;
  };
  double sa = 0.0;
  for (uint32_t i = threadIdx.x; i < n_above; i += kTpBlock) sa += exp_tang(D.d64(sh.above[i]), tab);
  double seg = 0.0;
  {
    double w = w0;
#pragma unroll 1
    for (int k = 0; k < kPer; ++k, w *= rho) seg += bin_mass(b0 + k, w);
  }
  // One exchange gives the totals of sa and seg and the prefix of seg (the
  // same sums, in the same order, as block_sum2 and block_exclusive_scan).
  const int lane = static_cast<int>(threadIdx.x % kWave), wv = static_cast<int>(threadIdx.x / kWave);
  double incl = seg;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const double t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  {
    const double sa_w = wave_sum_d(sa), seg_w = wave_sum_d(seg);
    if (lane == 0) {
      sh.loc.sa[wv] = sa_w;
      sh.loc.seg[wv] = seg_w;
    }
    if (lane == kWave - 1) sh.loc.scan[wv] = incl;
    if (threadIdx.x == 0) {
      sh.hb_lo = kHB - 1;
      sh.hb_hi = kHB - 1;
    }
  }
  __syncthreads();
  double tot = 0.0, base = 0.0;
  sa = 0.0;
  for (int k = 0; k < kNW; ++k) {
    sa += sh.loc.sa[k];
    tot += sh.loc.seg[k];
  }
  for (int k = 0; k < wv; ++k) base += sh.loc.scan[k];
  tot += sa;
  const double t_lo = static_cast<double>(P) * tot * (1.0 - kWinMargin);
  const double t_hi = static_cast<double>(P) * tot * (1.0 + kWinMargin);
  const double before = sa + (base + incl - seg);
  {
    // this thread's first bins where the running mass reaches t_lo and t_hi
    int k_lo = kHB, k_hi = kHB;
    double c = before;
    double w = w0;
#pragma unroll 1
    for (int k = 0; k < kPer; ++k, w *= rho) {
      c += bin_mass(b0 + k, w);
      if (k_lo == kHB && c >= t_lo) k_lo = b0 + k;
      if (k_hi == kHB && c >= t_hi) k_hi = b0 + k;
    }
    // bins grow with the thread index: a wave's smallest candidate is that
    // of its first lane that has one
    const uint64_t m_lo = __ballot(k_lo < kHB);
    const uint64_t m_hi = __ballot(k_hi < kHB);
    const int f_lo = __shfl(k_lo, m_lo ? static_cast<int>(__builtin_ctzll(m_lo)) : 0);
    const int f_hi = __shfl(k_hi, m_hi ? static_cast<int>(__builtin_ctzll(m_hi)) : 0);
    if (threadIdx.x % kWave == 0) {
      if (m_lo) atomicMin(&sh.hb_lo, f_lo);
      if (m_hi) atomicMin(&sh.hb_hi, f_hi);
    }
  }
  __syncthreads();
  Window W;
  W.b_lo = sa >= t_lo ? -1 : sh.hb_lo;  // -1: the list above the bins
  W.b_hi = sa >= t_hi ? -1 : sh.hb_hi;
  uint32_t inwin = 0, above = 0;
  double sb = 0.0, sb_max = 0.0;
  {
    double w = w0;
#pragma unroll 1
    for (int k = 0; k < kPer; ++k, w *= rho) {
      const int b = b0 + k;
      const uint32_t cnt = static_cast<uint32_t>(sh.u.hs.bins[b] >> kCountShift);
      if (b < W.b_lo) {
        above += cnt;
      } else if (b <= W.b_hi) {
        inwin += cnt;
      } else if (cnt) {  // below the window: the estimate and a bound on its error
        sb += bin_mass(b, w);
        sb_max += static_cast<double>(cnt) * w;
      }
    }
  }
  // Sparse pass when few lanes have three buckets reaching the window: a
  // bucket can reach it only if its maximum does (bf falls with z).
  auto reaches = [&](float x) { return fmaf(x, hk.kz4, hk.k04) < static_cast<float>(W.b_hi + 1) * kOffQ; };
  const bool full = reaches(tk.b3);
  const int64_t s1 = (tk.b1v >= 0 && reaches(tk.b1)) ? tk.b1v : -1;
  const int64_t s2 = (tk.b2v >= 0 && reaches(tk.b2)) ? tk.b2v : -1;
  {  // one exchange for the counts, the lanes with a third bucket reaching the window and the sums below it
    const uint32_t inwin_w = wave_sum_u(inwin), above_w = wave_sum_u(above), full_w = wave_sum_u(full ? 1u : 0u);
    const double sb_w = wave_sum_d(sb), sbm_w = wave_sum_d(sb_max);
    if (lane == 0) {
      sh.loc.u[0][wv] = inwin_w;
      sh.loc.u[1][wv] = above_w;
      sh.loc.u[2][wv] = full_w;
      sh.loc.d[0][wv] = sb_w;
      sh.loc.d[1][wv] = sbm_w;
    }
  }
  __syncthreads();  // also: every bin is read before the table below overwrites them
  inwin = above = 0u;
  uint32_t n_full = 0u;
  sb = sb_max = 0.0;
  for (int k = 0; k < kNW; ++k) {
    inwin += sh.loc.u[0][k];
    above += sh.loc.u[1][k];
    n_full += sh.loc.u[2][k];
    sb += sh.loc.d[0][k];
    sb_max += sh.loc.d[1][k];
  }
  W.inwin = inwin + (W.b_lo < 0 ? n_above : 0u);
  W.above = above + (W.b_lo >= 0 ? n_above : 0u);  // counts are exact
  W.s_below = sb;
  W.s_below_err = kBinMassRelErr * 1.01 * sb_max;  // 1.01: a logit's mass is below 1.0093 w_b
  if (W.inwin > static_cast<uint32_t>(kCap)) return false;
  // The counts are consumed: the same LDS now holds exp(centre of bin b - M).
  // A logit of bin b is exp(dd) = wtab[b] * exp(r), r = dd - centre, |r| at
  // most half a bin (0.0092 nats) plus the float32 rounding of bf (see
  // above): the degree-5 Taylor polynomial 1 + r + r^2 / 2 + r^3 c(r), c(r)
  // = 1/6 + r/24 + r^2/120 taken in float32 (its rounding, below 1.5e-8,
  // moves the polynomial by less than |r|^3 1.5e-8 < 3e-14; the remainder
  // r^6 / 720 is below 4.2e-15). The list takes the table-driven exp.
  const double lead0 = (static_cast<double>(A0) - static_cast<double>(D.M)) * D.invT64 + kHAbove;
  const double c0 = lead0 - 0.5 * invK;  // centre of bin b: c0 - b * invK
  {
    double w = exp(fma(-static_cast<double>(b0), invK, c0));
    const double rk = exp(-invK);
#pragma unroll 1
    for (int k = 0; k < kPer; ++k, w *= rk) sh.u.wtab[b0 + k] = w;
  }
  __syncthreads();

  if (n_full <= kSparseFullLanes &&
      exact_cut<Tin, true>(row, V, h, nvec, D, P, hk, sh, W, c0, invK, full, s1, s2, nuc))
    return true;
  if (approx_cut<Tin>(row, V, h, nvec, D, P, A0, hk, sh, W, nuc)) return true;
  return exact_cut<Tin, false>(row, V, h, nvec, D, P, hk, sh, W, c0, invK, true, -1, -1, nuc);
}

}  // namespace

// The first pass of a row without a nucleus (P >= 1, or a rejected P or
// temperature): the plain scan with its sums of 2^x, and the top-K hook
// (no histogram). Kept out of line, so that the kernel body around the
// nucleus path stays compact; its state goes in and comes back by value, so
// that no address of the kernel's scan state (lane, prefetched vectors,
// histogram hook) escapes into a call, which would move that state into
// private memory for the nucleus path too.
template <int LD>
struct Prefetched {
  vec4u v[LD];
};
template <typename HookB>
struct PlainResult {
  Lane L;
  HookB hb;
};
template <typename Tin, int LD, typename HookB>
__device__ __noinline__ PlainResult<HookB> plain_pass(const void* row, int32_t V, int64_t nvec, RowCtx cx, Lane L,
                                                      Prefetched<LD> pre, HookB hb) {
  scan_stretch<Tin, kTpBlock, 2, LD, false, true>(row, V, 0, nvec, true, true, nvec, cx, L, pre.v, hb);
  return PlainResult<HookB>{L, hb};
}

// LDS of the top-K selection, inside the window buffer (unused until the
// nucleus is computed) except for the result.
__device__ __forceinline__ topk::Lds topk_lds(TpShared& sh) {
  static_assert(2144 <= kCap, "top-K scratch fits in the window buffer");
  float* w = sh.win;
  topk::Lds s;
  s.key = reinterpret_cast<uint32_t*>(w);                // 1024 keys
  s.tag = reinterpret_cast<uint16_t*>(w + 1024);         // 1024 tags
  s.hist = reinterpret_cast<uint32_t*>(w + 1536);        // 512
  s.small_key = reinterpret_cast<uint32_t*>(w + 2048);   // 32
  s.small_tag = reinterpret_cast<uint16_t*>(w + 2080);   // 32
  s.misc = reinterpret_cast<uint32_t*>(w + 2112);        // 8
  s.red = reinterpret_cast<uint32_t*>(w + 2120);         // 8
  s.fail = reinterpret_cast<uint64_t*>(w + 2128);        // 8
  s.top = sh.topk;
  s.cap = 1024;
  return s;
}

// Finalises row r (wave 0 of the workgroup): its features and, in a
// streaming step (slot ids given), the token's join to its request slot:
// count, sums, minima and history, or the P-square markers.
__device__ __forceinline__ void finish_row(const RowArgs& a, int64_t r, const Partial& p, const RowCtx& cx,
                                           uint32_t fix, const Nucleus* nuc) {
  if (threadIdx.x >= kWave) return;
  p2::RowMarkers pm;
  pm.fetch(a, r);
  float conf[4];
  if (threadIdx.x == 0) {
    finalize_row(a, r, p, cx, fix, conf, nuc);
    stream_update(a.st, slot_load(a, r), conf);
  }
  if (pm.slot >= 0) p2::feed_row(a, pm, conf);
}

// SEQ: also the row's K largest logits (found in the stats pass) and row r
// of the verifier input sequence X, with the top-K probabilities taken on the
// renormalised nucleus.
template <typename Tin, bool SEQ>
__global__ __launch_bounds__(kTpBlock) __attribute__((amdgpu_waves_per_eu(4))) void topp_kernel(RowArgs a) {
  __shared__ TpShared sh;
  const int64_t r = blockIdx.x;
  if (r >= a.n_rows) return;
  constexpr int VEC = Elem<Tin>::kVec;
  const void* row = static_cast<const Tin*>(a.logits) + r * a.row_stride;
  const int64_t h = head_elems<Tin>(row, a.V);
  const int64_t nvec = (a.V - h) / VEC;
  constexpr int kLD = first_pass_depth<Tin>();  // with double buffering, kLD to 2 kLD loads in flight
  vec4u v[kLD];
  stretch_prefetch<Tin, kTpBlock, kLD>(row, h, 0, nvec, v);
  const RowCtx cx = row_ctx<Tin>(a, r, row);

  // Anchor of the histogram: the largest of the prefetched logits. The
  // histogram and the list are cleared meanwhile.
  float pm = -INFINITY;
#pragma unroll
  for (int u = 0; u < kLD; ++u) {
    float z[VEC];
    Elem<Tin>::unpack(v[u], z);
#pragma unroll
    for (int k = 0; k < VEC; ++k) pm = fmaxf(pm, z[k]);
  }
  pm = wave_max(pm);
  for (int b = threadIdx.x; b < kHB; b += kTpBlock) sh.u.hs.bins[b] = 0;
  if (threadIdx.x < 64) sh.exptab[threadIdx.x] = exp2(static_cast<double>(threadIdx.x) * (1.0 / 64.0));
  if (threadIdx.x == 0) sh.n_above = 0;
  if (threadIdx.x % kWave == 0) sh.red_f[threadIdx.x / kWave] = pm;
  __syncthreads();
  float A0 = sh.red_f[0];
  for (int k = 1; k < kNW; ++k) A0 = fmaxf(A0, sh.red_f[k]);
  // A row whose nucleus is computed (0 < P < 1, valid temperature) takes its
  // distribution from the float64 sums of the nucleus, so its first pass
  // forms no exps; any other row gets the plain features and no histogram.
  const float Prow = a.top_p[r];
  const bool nucleus_row = Prow > 0.0f && Prow < 1.0f && temperature_ok(cx.T);
  const bool anchored = nucleus_row && A0 > -INFINITY && A0 < INFINITY;
  const float invT = 1.0f / cx.T;
  // The top-K hook keeps each lane's three largest bucket maxima and the
  // steps of the first two: the sparse exact pass reads those buckets back
  // (and the sequence variant selects the K largest logits from them).
  HookPair<HistHook, topk::Hook> hp;
  HistHook& hk = hp.a;
  hp.b.init();
  hk.bins = sh.u.hs.bins;
  hk.above = sh.above;
  hk.n_above = &sh.n_above;
  hk.kz = anchored ? -invT * kHK : 0.0f;
  hk.k0 = anchored ? fmaf(A0, invT * kHK, kHAbove * kHK) : INFINITY;  // unanchored: nothing binned
  hk.kz4 = hk.kz * kOffQ;
  hk.k04 = hk.k0 * kOffQ;

  // 1. stats pass, building the histogram (S and E of the merged state are
  // only formed for a row without a nucleus)
  Lane L;
  lane_init(L);
  if (nucleus_row) {
    [[clang::always_inline]] scan_stretch<Tin, kTpBlock, 2, kLD, false, false>(row, a.V, 0, nvec, true, true, nvec,
                                                                               cx, L, v, hp);
  } else {
    Prefetched<kLD> pre;
#pragma unroll
    for (int u = 0; u < kLD; ++u) pre.v[u] = v[u];
    const auto res = plain_pass<Tin>(row, a.V, nvec, cx, L, pre, hp.b);
    L = res.L;
    hp.b = res.hb;
  }
  Partial p = block_merge<kTpBlock>(L, cx.c);
  const uint32_t fix = rank_fixup<Tin, kTpBlock>(row, a.V, nvec, cx);
  if constexpr (SEQ) {
    [[clang::always_inline]] topk::select_topk<Tin, kTpBlock, 2>(row, a.V, cx.h, 0, nvec, nvec, a.top_k, hp.b,
                                                                 topk_lds(sh));
    // the selection's scratch (the window buffer) is free again
  }
  if (threadIdx.x == 0) {
    sh.p = p;
    sh.fix = fix;
    sh.active = nucleus_row && (row_flags(a, r, p, cx.T) & (PR_FLAG_NONFINITE | PR_FLAG_BAD_TP)) == 0;
  }
  __syncthreads();
  p = sh.p;
  if (!sh.active) {
    if constexpr (SEQ) {
      if (threadIdx.x < kWave) {
        const float H = topk::topk_entropy_f32(sh.topk, a.top_k, p.m, cx.c, p.S);
        const float rho = topk::position_fraction(a.offsets, a.n_req, r);
        if (threadIdx.x == 0) {
          float conf[4];
          const uint32_t flags = finalize_row(a, r, p, cx, fix, conf);
          write_sequence_row(a, r, conf, flags, H, rho);
        }
      }
      return;
    }
    finish_row(a, r, p, cx, fix, nullptr);
    return;
  }

  const float T = cx.T;
  Dist D;
  D.M = p.m;
  D.invT = 1.0f / T;
  D.invT64 = 1.0 / static_cast<double>(T);
  const float P = Prow;
  Nucleus nuc;
  if (!(anchored && hist_nucleus<Tin>(row, a.V, cx.h, nvec, D, P, A0, hk, hp.b, sh, nuc)))
    nuc = legacy_nucleus<Tin>(row, a.V, cx.h, nvec, D, P, sh);
  if constexpr (SEQ) {
    if (threadIdx.x < kWave) {
      const int j = a.top_k < nuc.k ? a.top_k : nuc.k;  // the nucleus may hold fewer than K tokens
      const float H = topk::topk_entropy_f64(sh.topk, j, p.m, T, nuc.S);
      const float rho = topk::position_fraction(a.offsets, a.n_req, r);
      if (threadIdx.x == 0) {
        float conf[4];
        const uint32_t flags = finalize_row(a, r, p, cx, fix, conf, &nuc);
        write_sequence_row(a, r, conf, flags, H, rho);
      }
    }
    return;
  }
  finish_row(a, r, p, cx, fix, &nuc);
}

size_t topp_workspace(pr_dtype, int64_t, int32_t) { return 0; }

hipError_t launch_topp(const RowArgs& a, pr_dtype dtype, void*, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(a.n_rows));
  const bool seq = a.X != nullptr;
  if (dtype == PR_BF16) {
    if (seq)
      topp_kernel<uint16_t, true><<<grid, kTpBlock, 0, stream>>>(a);
    else
      topp_kernel<uint16_t, false><<<grid, kTpBlock, 0, stream>>>(a);
  } else {
    if (seq)
      topp_kernel<float, true><<<grid, kTpBlock, 0, stream>>>(a);
    else
      topp_kernel<float, false><<<grid, kTpBlock, 0, stream>>>(a);
  }
  return hipGetLastError();
}

}  // namespace pr
