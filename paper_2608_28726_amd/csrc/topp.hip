// Top-p (nucleus) features: the nucleus is the shortest prefix of the token
// order (larger logit first, equal logits by lower index) whose probability
// mass reaches P of the total, k = min{ j : C_j >= P * S }; the distribution
// features are then those of the renormalised nucleus (the per-token
// features of Pro-Router, Sec. 3.1, Eq. 3, after top-p truncation).
//
// One 512-thread workgroup per row, at most five reads of the row:
//  1. the stats pass of the row kernel (max M, rank of y, argmax, margin);
//  2. a 4096-bin histogram over the distance (M - z) / T in nats of every
//     logit within 50 nats of M, with float64 masses exp((z - M) / T) and
//     counts in LDS, plus the float64 total S; its prefix sums give the
//     bins [b_lo, b_hi] in which the cumulative mass crosses P * S;
//  3. float64 sums over the bins above b_lo (mass, count, entropy term) and
//     the logits of the crossing bins gathered into LDS;
//  4. a bitonic sort of the gathered logits (descending) and a float64 scan
//     along it gives the exact k. Logits beyond 50 nats can never be in a
//     nucleus with P < 1 (their total mass is below V * e^-50 of S).
// When the crossing bins hold more than 4096 logits, a byte-wise radix
// refinement over order-preserving keys (four more reads) finds the boundary
// value instead; equal logits have equal mass, so ties are resolved by
// counting.
#include "topp.h"

#include "row_scan.h"

namespace pr {

using namespace scan;

namespace {

constexpr int kTpBlock = 512;
constexpr int kBins = 4096;
constexpr float kDMax = 50.0f;  // nats below the maximum
constexpr int kCap = 4096;      // gathered logits sorted in LDS
constexpr int kNW = kTpBlock / kWave;

struct TpShared {
  double mass[kBins];
  uint32_t cnt[kBins];
  float win[kCap];
  double red_d[2][kNW];
  uint32_t red_u[kNW];
  double S64, target, massAbove, Eabove, SN, EN;
  uint32_t b_lo, b_hi, wcount, cntAbove, jfirst, rcount;
  int32_t active;
  Partial p;
  uint32_t fix;
  // radix refinement
  double rmass[256], rE[256];
  uint32_t rcnt[256];
  uint32_t prefix, rdigit;
};

// Calls fn(z) for every logit of the row (order irrelevant).
template <typename Tin, typename Fn>
__device__ __forceinline__ void for_each_logit(const void* row, int32_t V, int64_t h, int64_t nvec, Fn fn) {
  constexpr int VEC = Elem<Tin>::kVec;
  const int t = threadIdx.x;
  if (t < h) fn(Elem<Tin>::load1(row, t));
  const vec4u* vp = reinterpret_cast<const vec4u*>(static_cast<const Tin*>(row) + h);
  for (int64_t i = t; i < nvec; i += kTpBlock) {
    float z[VEC];
    Elem<Tin>::unpack(vp[i], z);
#pragma unroll
    for (int k = 0; k < VEC; ++k) fn(z[k]);
  }
  for (int64_t e = h + nvec * VEC + t; e < V; e += kTpBlock) fn(Elem<Tin>::load1(row, e));
}

// Block-wide sums of (x, y) in a fixed order; every thread gets the result.
__device__ void block_sum2(double& x, double& y, TpShared& sh) {
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

__device__ uint32_t block_sum_u(uint32_t v, TpShared& sh) {
  v = wave_sum_u(v);
  __syncthreads();
  if (threadIdx.x % kWave == 0) sh.red_u[threadIdx.x / kWave] = v;
  __syncthreads();
  uint32_t tot = 0;
  for (int k = 0; k < kNW; ++k) tot += sh.red_u[k];
  __syncthreads();
  return tot;
}

// Exclusive block scan of one double per thread (thread order).
__device__ double block_exclusive_scan(double v, TpShared& sh) {
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

// Bitonic sort of sh.win[0..n2) into descending order (n2 a power of two).
__device__ void bitonic_desc(float* a, int n2) {
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
// cntAbove hold the exact sums of the logits above b_lo.
template <typename Tin>
__device__ Nucleus radix_boundary(const void* row, int32_t V, int64_t h, int64_t nvec, const Dist& D, TpShared& sh) {
  double massGT = sh.massAbove, EGT = sh.Eabove;
  uint32_t cntGT = sh.cntAbove;
  uint32_t prefix = 0, mask = 0, cnt_last = 0;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int b = threadIdx.x; b < 256; b += kTpBlock) {
      sh.rmass[b] = 0.0;
      sh.rE[b] = 0.0;
      sh.rcnt[b] = 0;
    }
    __syncthreads();
    const uint32_t blo = sh.b_lo, bhi = sh.b_hi;
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
      atomicAdd(&sh.rmass[dg], e);
      atomicAdd(&sh.rE[dg], e * dd);
      atomicAdd(&sh.rcnt[dg], 1u);
    });
    __syncthreads();
    if (threadIdx.x == 0) {
      int dg = 255;
      for (; dg > 0; --dg) {  // descending keys: larger logits first
        if (massGT + sh.rmass[dg] >= sh.target) break;
        massGT += sh.rmass[dg];
        EGT += sh.rE[dg];
        cntGT += sh.rcnt[dg];
      }
      sh.rdigit = static_cast<uint32_t>(dg);
      sh.massAbove = massGT;
      sh.Eabove = EGT;
      sh.cntAbove = cntGT;
      sh.rcount = sh.rcnt[dg];
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

}  // namespace

template <typename Tin>
__global__ __launch_bounds__(kTpBlock) void topp_kernel(RowArgs a) {
  __shared__ TpShared sh;
  const int64_t r = blockIdx.x;
  if (r >= a.n_rows) return;
  constexpr int VEC = Elem<Tin>::kVec;
  const void* row = static_cast<const Tin*>(a.logits) + r * a.row_stride;
  const int64_t h = head_elems<Tin>(row, a.V);
  const int64_t nvec = (a.V - h) / VEC;
  constexpr int kLD = 4;  // loads in flight per lane: 4 to 8 with double buffering
  vec4u v[kLD];
  stretch_prefetch<Tin, kTpBlock, kLD>(row, h, 0, nvec, v);
  const RowCtx cx = row_ctx<Tin>(a, r, row);

  // 1. stats pass
  Lane L;
  lane_init(L);
  scan_stretch<Tin, kTpBlock, 2, kLD>(row, a.V, 0, nvec, true, true, nvec, cx, L, v);
  Partial p = block_merge<kTpBlock>(L, cx.c);
  const uint32_t fix = rank_fixup<Tin, kTpBlock>(row, a.V, nvec, cx);
  if (threadIdx.x == 0) {
    sh.p = p;
    sh.fix = fix;
    const float P = a.top_p[r];
    sh.active = (row_flags(a, r, p, cx.T) & (PR_FLAG_NONFINITE | PR_FLAG_BAD_TP)) == 0 && P < 1.0f;
  }
  __syncthreads();
  p = sh.p;
  if (!sh.active) {
    if (threadIdx.x == 0) {
      float conf[4];
      finalize_row(a, r, p, cx, fix, conf);
    }
    return;
  }

  const float T = cx.T;
  Dist D;
  D.M = p.m;
  D.invT = 1.0f / T;
  D.invT64 = 1.0 / static_cast<double>(T);

  // 2. histogram of the candidates' masses over distance bins
  for (int b = threadIdx.x; b < kBins; b += kTpBlock) {
    sh.mass[b] = 0.0;
    sh.cnt[b] = 0;
  }
  if (threadIdx.x == 0) sh.wcount = 0;
  __syncthreads();
  double s64 = 0.0, unused = 0.0;
  for_each_logit<Tin>(row, a.V, cx.h, nvec, [&](float z) {
    const float d = D.nats(z);
    if (!(d < kDMax)) return;
    const double e = exp(D.d64(z));
    const int b = D.bin(d);
    atomicAdd(&sh.mass[b], e);
    atomicAdd(&sh.cnt[b], 1u);
    s64 += e;
  });
  block_sum2(s64, unused, sh);  // fixed-order total: deterministic
  const double target = static_cast<double>(a.top_p[r]) * s64;
  const double tol = 1e-9 * s64;

  // crossing bins: the first bins whose cumulative mass reaches target -/+ tol
  constexpr int kPer = kBins / kTpBlock;
  const int b0 = threadIdx.x * kPer;
  double seg = 0.0;
  for (int k = 0; k < kPer; ++k) seg += sh.mass[b0 + k];
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
      c += sh.mass[b0 + k];
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
    if (b < b_lo) above += sh.cnt[b];
    else if (b <= b_hi) inwin += sh.cnt[b];
  }
  above = block_sum_u(above, sh);
  inwin = block_sum_u(inwin, sh);

  // 3. exact sums above the crossing bins; gather the crossing bins' logits
  double mA = 0.0, eA = 0.0;
  const bool gather = inwin <= static_cast<uint32_t>(kCap);
  for_each_logit<Tin>(row, a.V, cx.h, nvec, [&](float z) {
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
    // 4. sort the crossing logits (descending) and scan their masses
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
    nuc = radix_boundary<Tin>(row, a.V, cx.h, nvec, D, sh);
  }
  if (threadIdx.x == 0) {
    float conf[4];
    finalize_row(a, r, p, cx, fix, conf, &nuc);
  }
}

size_t topp_workspace(pr_dtype, int64_t, int32_t) { return 0; }

hipError_t launch_topp(const RowArgs& a, pr_dtype dtype, void*, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(a.n_rows));
  if (dtype == PR_BF16)
    topp_kernel<uint16_t><<<grid, kTpBlock, 0, stream>>>(a);
  else
    topp_kernel<float><<<grid, kTpBlock, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace pr
