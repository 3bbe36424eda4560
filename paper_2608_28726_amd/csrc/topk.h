// The K largest logits of a row, for the top-K entropy of the paper's
// verifier input (Pro-Router, Sec. 3.1, Eq. 3 and the text after it:
// h_t = -H_t with H_t summed over the K = 20 most probable tokens). The
// row's other features come from the same single pass; this adds little to
// it (internal, device code only).
//
// During the scan every lane already keeps its largest and second largest
// bucket maximum (a bucket is one step's vectors of one lane, or one scalar
// head/tail logit) and the step of the largest; the hook below adds the
// third largest bucket maximum b3 and the step of the second. After the scan
// (select_topk):
//  1. theta_lb = the K-th largest lane maximum of the workgroup (a radix
//     select over the lanes' maxima). At least K logits are >= theta_lb and
//     fewer than K lanes have a maximum above it.
//  2. Those lanes read their largest bucket, and their second largest when
//     its maximum is above theta_lb, back from memory and list every logit
//     above theta_lb: at most 2(K-1) buckets, kept in LDS together with the
//     lane that listed them.
//  3. theta_c = the K-th largest listed logit (theta_lb when fewer than K
//     are listed). Every logit above theta_c is then listed, unless a lane's
//     third largest bucket maximum exceeds theta_c. Such a lane (rare: it
//     holds three of the largest logits) withdraws its entries and the
//     workgroup lists every logit of that lane above theta_c, compacting the
//     list to its K largest entries whenever it would overflow.
//  4. The K largest logits are the listed ones above the K-th largest listed
//     value v_K, and copies of v_K (ties have equal probability, so which of
//     them count does not matter); they are written to LDS in descending
//     order.
// All choices are made on order-preserving 32-bit keys of the raw logits, so
// the result is exact and does not depend on the launch shape.
#pragma once

#include "row_scan.h"

namespace pr {
namespace topk {

constexpr int kMaxK = 32;  // largest K supported

// Per-lane tracking during the scan (hook of scan_stretch). The lane's
// largest and second largest bucket maxima, and the step of the largest, are
// the scan's own t1, t2, t1v.
struct Hook {
  float b3;      // third largest bucket maximum
  int32_t b2v;   // step (first vector index) of the second, -1: a scalar bucket
  float b1, b2;  // the scan's t1, t2 at the end of the stretch
  int32_t b1v;   // the scan's t1v at the end of the stretch
  __device__ __forceinline__ void init() {
    b3 = -INFINITY;
    b2v = -1;
  }
  template <int N>
  __device__ __forceinline__ void step(const float (&)[N], const float (&)[N], float cmax, int64_t i,
                                       const scan::Lane& L) {
    const bool up1 = cmax > L.t1;
    const bool up2 = cmax > L.t2;
    b3 = __builtin_amdgcn_fmed3f(L.t2, b3, cmax);
    b2v = up1 ? L.t1v : (up2 ? static_cast<int32_t>(i) : b2v);
  }
  __device__ __forceinline__ void scalar(float z, float, int64_t, const scan::Lane& L) {
    const bool up1 = z > L.t1;
    const bool up2 = z > L.t2;
    b3 = __builtin_amdgcn_fmed3f(L.t2, b3, z);
    b2v = up1 ? L.t1v : (up2 ? -1 : b2v);
  }
  __device__ __forceinline__ void finish(const scan::Lane& L) {
    b1 = L.t1;
    b1v = L.t1v;
    b2 = L.t2;
  }
};

// Indices into Lds::misc.
enum { kN = 0, kNSmall, kTotal, kDigit, kNeed, kMisc };

// LDS used by select_topk. `top` receives the result and must outlive the
// call; everything else is scratch during the call.
struct Lds {
  uint32_t* key;        // [cap] listed logits as keys (0: withdrawn)
  uint16_t* tag;        // [cap] thread that listed each entry
  uint32_t* hist;       // [2][256] radix histograms
  uint32_t* small_key;  // [kMaxK] compaction buffer
  uint16_t* small_tag;  // [kMaxK]
  uint32_t* misc;       // [kMisc]
  uint32_t* red;        // [workgroup waves]
  uint64_t* fail;       // [workgroup waves]
  float* top;           // [kMaxK] result: the K largest logits, descending
  int cap;
};

// Capacity of the list: at least 2(K-1) buckets of 16 logits, and K plus one
// logit per thread (a compaction step).
template <int BLOCK>
constexpr int list_cap() {
  return BLOCK >= 1024 ? 2048 : 1024;
}

// Dedicated LDS for a workgroup of BLOCK threads.
template <int BLOCK>
struct Store {
  uint32_t key[list_cap<BLOCK>()];
  uint16_t tag[list_cap<BLOCK>()];
  uint32_t hist[2 * 256];
  uint32_t small_key[kMaxK];
  uint16_t small_tag[kMaxK];
  uint32_t misc[kMisc];
  uint32_t red[BLOCK / kWave];
  uint64_t fail[BLOCK / kWave];
  float top[kMaxK];
  __device__ Lds view() {
    return Lds{key, tag, hist, small_key, small_tag, misc, red, fail, top, list_cap<BLOCK>()};
  }
};

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int lane = __lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  return v;
}

// The j-th largest (1-based) of the keys that the threads of the workgroup
// pass to `keys` (each thread calls keys(fn) and fn(key) for each of its
// keys; zero keys are ignored). Radix select over 8-bit digits, most
// significant first; PASSES = 2 when every key's low 16 bits follow from its
// sign (keys of bfloat16 values). Returns 0 when there are fewer than j
// keys; *gt receives the number of keys above the result (all of them when
// fewer than j). Every thread calls it.
template <int BLOCK, int PASSES, typename Keys>
__device__ uint32_t select_desc(Keys&& keys, uint32_t j, const Lds& s, uint32_t* gt) {
  static_assert(PASSES == 2 || PASSES == 4, "digits of 8 bits over 16 or 32 key bits");
  uint32_t prefix = 0, mask = 0, need = j;
  for (int b = threadIdx.x; b < 256; b += BLOCK) s.hist[b] = 0;
  __syncthreads();
  for (int pass = 0; pass < PASSES; ++pass) {
    const int shift = 24 - 8 * pass;
    uint32_t* h = s.hist + (pass & 1) * 256;
    keys([&](uint32_t k) {
      if (k != 0u && (k & mask) == prefix) atomicAdd(&h[(k >> shift) & 255u], 1u);
    });
    if (pass + 1 < PASSES) {
      uint32_t* hn = s.hist + ((pass + 1) & 1) * 256;
      for (int b = threadIdx.x; b < 256; b += BLOCK) hn[b] = 0;
    }
    __syncthreads();
    if (threadIdx.x < kWave) {
      // lane l holds digits 255 - 4l .. 252 - 4l: descending order
      const int l = threadIdx.x;
      const uint32_t c0 = h[255 - 4 * l], c1 = h[254 - 4 * l], c2 = h[253 - 4 * l], c3 = h[252 - 4 * l];
      const uint32_t tot = c0 + c1 + c2 + c3;
      const uint32_t incl = wave_incl_scan(tot);
      const uint32_t excl = incl - tot;
      if (pass == 0 && l == kWave - 1) s.misc[kTotal] = incl;
      if (need > excl && need <= incl) {
        uint32_t r = need - excl, q = 0;
        if (r > c0) {
          r -= c0;
          q = 1;
          if (r > c1) {
            r -= c1;
            q = 2;
            if (r > c2) {
              r -= c2;
              q = 3;
            }
          }
        }
        s.misc[kDigit] = 255u - 4u * static_cast<uint32_t>(l) - q;
        s.misc[kNeed] = r;
      }
    }
    __syncthreads();
    if (pass == 0) {
      const uint32_t total = s.misc[kTotal];
      if (total < j) {
        *gt = total;
        return 0u;
      }
    }
    prefix |= s.misc[kDigit] << shift;
    need = s.misc[kNeed];
    mask |= 255u << shift;
  }
  if (PASSES == 2) prefix |= (prefix & 0x80000000u) ? 0u : 0xffffu;
  *gt = j - need;
  return prefix;
}

// Number of listed keys above kth (every thread gets it).
template <int BLOCK>
__device__ uint32_t count_above(const Lds& s, uint32_t n, uint32_t kth) {
  uint32_t c = 0;
  for (uint32_t e = threadIdx.x; e < n; e += BLOCK) c += s.key[e] > kth ? 1u : 0u;
  c = wave_sum_u(c);
  __syncthreads();
  if (__lane_id() == 0) s.red[threadIdx.x / kWave] = c;
  __syncthreads();
  uint32_t tot = 0;
  for (int w = 0; w < BLOCK / kWave; ++w) tot += s.red[w];
  __syncthreads();
  return tot;
}

// Keeps the listed keys above kth (fewer than kMaxK of them) and drops the
// rest. Returns the new list length.
template <int BLOCK>
__device__ uint32_t compact(const Lds& s, uint32_t n, uint32_t kth) {
  if (threadIdx.x == 0) s.misc[kNSmall] = 0;
  __syncthreads();
  for (uint32_t e = threadIdx.x; e < n; e += BLOCK) {
    if (s.key[e] > kth) {
      const uint32_t p = atomicAdd(&s.misc[kNSmall], 1u);
      if (p < static_cast<uint32_t>(kMaxK)) {
        s.small_key[p] = s.key[e];
        s.small_tag[p] = s.tag[e];
      }
    }
  }
  __syncthreads();
  const uint32_t ns = min(s.misc[kNSmall], static_cast<uint32_t>(kMaxK));
  for (uint32_t e = threadIdx.x; e < ns; e += BLOCK) {
    s.key[e] = s.small_key[e];
    s.tag[e] = s.small_tag[e];
  }
  if (threadIdx.x == 0) s.misc[kN] = ns;
  __syncthreads();
  return ns;
}

// The K largest logits of a row scanned by one workgroup (vector index range
// [vb, ve) of the row's nvec aligned vectors, h scalar head logits, the tail
// after them), written to s.top in descending order (-inf where the row has
// fewer than K logits). hk is the lane's hook after the scan; U vectors per
// step. Every thread of the workgroup calls it.
template <typename Tin, int BLOCK, int U>
__device__ void select_topk(const void* row, int32_t V, int64_t h, int64_t vb, int64_t ve, int64_t nvec, int K,
                            const Hook& hk, const Lds& s) {
  constexpr int VEC = Elem<Tin>::kVec;
  constexpr int PASSES = sizeof(Tin) == 2 ? 2 : 4;
  constexpr int NW = BLOCK / kWave;
  static_assert(U * VEC <= 16, "at most 16 logits per bucket");
  static_assert(2 * (kMaxK - 1) * 16 <= list_cap<BLOCK>() && kMaxK + BLOCK <= list_cap<BLOCK>(),
                "list capacity");
  const uint32_t Ku = static_cast<uint32_t>(K);
  const vec4u* vp = reinterpret_cast<const vec4u*>(static_cast<const Tin*>(row) + h);
  const int t = threadIdx.x;
  const uint32_t cap = static_cast<uint32_t>(s.cap);

  // 1. theta_lb: the K-th largest lane maximum (a row with NaN may leave
  // fewer than K non-zero keys; nothing is listed then).
  uint32_t gt = 0;
  const uint32_t k1 = float_key(hk.b1);
  uint32_t klb = select_desc<BLOCK, PASSES>([&](auto fn) { fn(k1); }, Ku, s, &gt);
  if (klb == 0u) klb = 0xffffffffu;

  // 2. list the logits above theta_lb of the lanes' two largest buckets
  if (t == 0) s.misc[kN] = 0;
  __syncthreads();
  auto append = [&](uint32_t k, int owner) {
    const uint32_t p = atomicAdd(&s.misc[kN], 1u);
    if (p < cap) {
      s.key[p] = k;
      s.tag[p] = static_cast<uint16_t>(owner);
    }
  };
  auto list_bucket = [&](float bmax, int32_t bv) {
    if (!(float_key(bmax) > klb)) return;
    if (bv < 0) {  // a scalar bucket holds its maximum only
      append(float_key(bmax), t);
      return;
    }
    for (int u = 0; u < U; ++u) {
      const int64_t j = static_cast<int64_t>(bv) + static_cast<int64_t>(u) * BLOCK;
      if (j >= ve) break;
      float z[VEC];
      Elem<Tin>::unpack(vp[j], z);
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        const uint32_t kz = float_key(z[k]);
        if (kz > klb) append(kz, t);
      }
    }
  };
  list_bucket(hk.b1, hk.b1v);
  list_bucket(hk.b2, hk.b2v);
  __syncthreads();
  uint32_t n = min(s.misc[kN], cap);  // <= 2 (K - 1) * 16 <= cap: fewer than K lanes list

  // 3. theta_c, and the lanes whose third bucket may hold more
  uint32_t kc = klb, gtc = n;
  if (n >= Ku) kc = select_desc<BLOCK, PASSES>([&](auto fn) {
      for (uint32_t e = t; e < n; e += BLOCK) fn(s.key[e]);
    }, Ku, s, &gtc);
  const bool fail = float_key(hk.b3) > kc && kc != 0xffffffffu;
  uint32_t kK = kc, gtK = gtc;
  if (__syncthreads_or(fail)) {
    const uint64_t m = __ballot(fail);
    if (__lane_id() == 0) s.fail[t / kWave] = m;
    __syncthreads();
    const int64_t tail0 = h + nvec * VEC;
    // One withdrawn-and-relisted lane at a time, the whole workgroup reading
    // that lane's vectors. add() lists z when above kc (one call per thread,
    // workgroup-uniform), compacting first when the list would overflow.
    auto add = [&](float z, int owner) {
      bool c = float_key(z) > kc;
      const uint32_t tot = static_cast<uint32_t>(__syncthreads_count(c));
      if (tot == 0) return;
      if (n + tot > cap) {
        uint32_t g = 0;
        const uint32_t sel = select_desc<BLOCK, PASSES>([&](auto fn) {
            for (uint32_t e = t; e < n; e += BLOCK) fn(s.key[e]);
          }, Ku, s, &g);
        if (sel > kc) kc = sel;
        n = compact<BLOCK>(s, n, kc);
        c = float_key(z) > kc;
      }
      if (c) append(float_key(z), owner);
      __syncthreads();
      n = min(s.misc[kN], cap);
    };
    for (int w = 0; w < NW; ++w) {
      uint64_t fm = s.fail[w];
      while (fm) {
        const int tf = w * kWave + (__ffsll(static_cast<long long>(fm)) - 1);
        fm &= fm - 1;
        for (uint32_t e = t; e < n; e += BLOCK)
          if (s.tag[e] == tf) s.key[e] = 0u;
        __syncthreads();
        const int64_t first = vb + tf;
        const int64_t nv = first < ve ? (ve - first + BLOCK - 1) / BLOCK : 0;
        for (int64_t base = 0; base < nv; base += BLOCK) {
          const int64_t sidx = base + t;
          float z[VEC];
          if (sidx < nv) {
            Elem<Tin>::unpack(vp[first + sidx * BLOCK], z);
          } else {
#pragma unroll
            for (int k = 0; k < VEC; ++k) z[k] = -INFINITY;
          }
          uint32_t cnt = 0;
#pragma unroll
          for (int k = 0; k < VEC; ++k) cnt += float_key(z[k]) > kc ? 1u : 0u;
          cnt = wave_sum_u(cnt);
          if (__lane_id() == 0) s.red[t / kWave] = cnt;
          __syncthreads();
          uint32_t tot = 0;
          for (int q = 0; q < NW; ++q) tot += s.red[q];
          if (n + tot <= cap) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
              const uint32_t kz = float_key(z[k]);
              if (kz > kc) append(kz, tf);
            }
            __syncthreads();
            n = min(s.misc[kN], cap);
          } else {
#pragma unroll
            for (int k = 0; k < VEC; ++k) add(z[k], tf);
          }
        }
        // the lane's scalar head and tail logits
        float zh = -INFINITY, zt = -INFINITY;
        if (t == 0) {
          if (tf < h) zh = Elem<Tin>::load1(row, tf);
          if (tail0 + tf < V) zt = Elem<Tin>::load1(row, tail0 + tf);
        }
        add(zh, tf);
        add(zt, tf);
      }
    }
    // 4. the K-th largest listed value, never below theta_c
    uint32_t g = 0;
    const uint32_t sel = select_desc<BLOCK, PASSES>([&](auto fn) {
        for (uint32_t e = t; e < n; e += BLOCK) fn(s.key[e]);
      }, Ku, s, &g);
    if (sel != 0u && sel >= kc) {
      kK = sel;
      gtK = g;
    } else {
      kK = kc;
      gtK = count_above<BLOCK>(s, n, kc);
    }
  }

  // 4. the gtK listed logits above kK, sorted, then copies of kK
  if (t == 0) s.misc[kNSmall] = 0;
  __syncthreads();
  for (uint32_t e = t; e < n; e += BLOCK) {
    if (s.key[e] > kK) {
      const uint32_t p = atomicAdd(&s.misc[kNSmall], 1u);
      if (p < static_cast<uint32_t>(kMaxK)) s.small_key[p] = s.key[e];
    }
  }
  __syncthreads();
  if (gtK > static_cast<uint32_t>(K)) gtK = static_cast<uint32_t>(K);  // cannot happen: fewer than K above kK
  if (t < K) {
    if (static_cast<uint32_t>(t) < gtK) {
      const uint32_t mine = s.small_key[t];
      uint32_t rank = 0;
      for (uint32_t q = 0; q < gtK; ++q) {
        const uint32_t o = s.small_key[q];
        rank += (o > mine || (o == mine && q < static_cast<uint32_t>(t))) ? 1u : 0u;
      }
      s.top[rank] = key_float(mine);
    } else {
      s.top[t] = key_float(kK);
    }
  }
  __syncthreads();
}

// -sum over the j largest logits top[0..j) of p log p with
// p = 2^x / S, x = (z - M) * log2(e) / T in the row state's reference
// (A = round(M c), delta = M c - A, S relative to M c): the float32 path of
// a row without a nucleus. Called by the 64 lanes of one wave (j <= 64);
// every lane gets the sum.
__device__ __forceinline__ float topk_entropy_f32(const float* top, int j, float M, float c, float S_raw) {
  const float A = M * c;
  const float delta = fmaf(M, c, -A);
  const float S = S_raw * fast_exp2(-delta);
  const float lnS = ln_sum(S);
  float term = 0.0f;
  const int l = __lane_id();
  if (l < j) {
    const float z = top[l];
    if (z != -INFINITY) {
      const float x = fmaf(z, c, -A) - delta;
      const float p = fast_exp2(x) / S;
      term = p * (kLn2 * x - lnS);
    }
  }
  return -wave_sum(term);
}

// The same over a nucleus: p = exp((z - M) / T) / S_N in float64.
__device__ __forceinline__ float topk_entropy_f64(const float* top, int j, float M, float T, double S_N) {
  const double lnS = ln_sum(S_N);
  double term = 0.0;
  const int l = __lane_id();
  if (l < j) {
    const float z = top[l];
    if (z != -INFINITY) {
      const double d = (static_cast<double>(z) - static_cast<double>(M)) / static_cast<double>(T);
      const double p = exp(d) / S_N;
      term = p * (d - lnS);
    }
  }
  return static_cast<float>(-wave_sum_d(term));
}

// Position fraction t / T of row r within its request: request i owns rows
// offsets[i] .. offsets[i+1]-1 (non-decreasing offsets, offsets[0] <= r <
// offsets[n_req]). A 64-ary search by one wave; every lane gets the result
// (NaN when r lies outside the offsets).
__device__ __forceinline__ float position_fraction(const int32_t* offsets, int32_t n_req, int64_t r) {
  const int lane = __lane_id();
  int64_t lo = 0, span = n_req;  // answer in [lo, lo + span)
  while (span > kWave) {
    const int64_t step = (span + kWave - 1) / kWave;
    const int64_t k = static_cast<int64_t>(lane) * step;
    const bool le = k < span && offsets[lo + k] <= r;
    const int cnt = __popcll(__ballot(le));
    if (cnt == 0) return __uint_as_float(0x7fc00000u);
    lo += static_cast<int64_t>(cnt - 1) * step;
    span = step < n_req - lo ? step : n_req - lo;
  }
  const bool le = lane < span && offsets[lo + lane] <= r;
  const int cnt = __popcll(__ballot(le));
  if (cnt == 0) return __uint_as_float(0x7fc00000u);
  const int64_t i = lo + cnt - 1;
  const int32_t o0 = offsets[i], o1 = offsets[i + 1];
  if (r >= o1) return __uint_as_float(0x7fc00000u);
  return static_cast<float>(static_cast<double>(r - o0 + 1) / static_cast<double>(o1 - o0));
}

}  // namespace topk
}  // namespace pr
