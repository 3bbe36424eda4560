// Vocabulary-row reduction: per-token confidence features in one pass over
// each logit row (Pro-Router, Sec. 3.1, Eq. 3, extended to max logit,
// logsumexp, entropy, log-probability, top-1/top-2 margin and rank of the
// sampled token, after temperature).
//
// One or more workgroups stream a row with 16-byte loads. Every lane keeps
// an online (max, sum 2^x, sum 2^x * x) state in base 2 with exponent
// argument x = z * log2(e)/T - a (a = the lane's running max times
// log2(e)/T), the top-1 value/index and top-2 value, and the number of
// tokens that precede the sampled token y in the order "larger logit first,
// equal logits by lower index". Comparisons use the raw logits, so
// temperature scaling cannot create false ties. Lanes merge with wave
// shuffles, waves through LDS; a row split over G workgroups merges the G
// partial states either in a second kernel or in the last workgroup to
// finish (streaming decode).
#include "row_features.h"

namespace pr {

namespace {

struct Lane {
  float mw;        // running max of the wave's logits (wave-uniform in the vector loop)
  float a;         // reference of S and E: mw * c, or kNegSentinel
  float S0, S1;    // two accumulators of sum 2^x (alternating elements)
  float E0, E1;    // two accumulators of sum 2^x * x
  float t1, t2;    // largest and second value this lane recorded
  int32_t t1i;     // index of t1 (lowest among ties)
  uint32_t cnt;    // rank counts (ballot totals are added in lane 0 only)
  float thr2;      // wave-uniform: max over the wave's lanes of t2
};

struct RowCtx {
  float c;           // log2(e) / T
  float zy;          // logit of the sampled token (NaN when y is invalid)
  float thr_before;  // strict threshold for vectors wholly before y
  float thr_lo;      // min of the two thresholds: lazy-skip test
  int32_t y;         // sampled id, or -1 when invalid
  int64_t h;         // scalar head elements before the first aligned vector
};

__device__ __forceinline__ void lane_init(Lane& L) {
  L.mw = -INFINITY;
  L.a = kNegSentinel;
  L.S0 = L.S1 = L.E0 = L.E1 = 0.0f;
  L.t1 = -INFINITY;
  L.t2 = -INFINITY;
  L.t1i = kNoIndex;
  L.cnt = 0;
  L.thr2 = -INFINITY;
}

// Moves the lane's reference up to a_new = m_new * c (m_new >= the old max).
__device__ __forceinline__ void lane_rescale(Lane& L, float m_new, float c) {
  L.mw = m_new;
  const float a_new = m_new * c;
  const float d = fmaxf(L.a - a_new, -kBig);
  const float s = fast_exp2(d);
  const float sd = s * d;
  L.E0 = fmaf(sd, L.S0, s * L.E0);
  L.E1 = fmaf(sd, L.S1, s * L.E1);
  L.S0 *= s;
  L.S1 *= s;
  L.a = a_new;
}

// NV vectors of one lane; vector u has vector index i + u * BLOCK. Every lane
// of the wave calls this together (wave-uniform control flow), so the
// cross-lane steps below see all 64 lanes.
template <typename Tin, int NV, int BLOCK>
__device__ __forceinline__ void consume(const uint4 (&v)[NV], int64_t i, const RowCtx& cx, Lane& L) {
  constexpr int VEC = Elem<Tin>::kVec;
  float z[NV * VEC];
#pragma unroll
  for (int u = 0; u < NV; ++u) Elem<Tin>::unpack(v[u], z + u * VEC);

  float cmax = z[0];
#pragma unroll
  for (int k = 1; k < NV * VEC; ++k) cmax = fmaxf(cmax, z[k]);

  // The wave shares one reference, its running maximum: every exponent
  // argument stays <= 0 and the reference moves only on a new wave maximum.
  if (__any(cmax > L.mw)) lane_rescale(L, wave_max(cmax), cx.c);

  // Top-1/top-2. An element no larger than thr2 cannot change the row's
  // result: some lane already holds two values >= it at lower indices (every
  // chunk lies above the previous ones in index order). thr2 rises quickly,
  // so the per-element update below runs on few chunks.
  if (__any(cmax > L.thr2)) {
    if (cmax > L.t2) {
#pragma unroll
      for (int u = 0; u < NV; ++u) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
          const float zk = z[u * VEC + k];
          if (zk > L.t1) {
            L.t2 = L.t1;
            L.t1 = zk;
            L.t1i = static_cast<int32_t>(cx.h + (i + u * BLOCK) * VEC + k);
          } else if (zk > L.t2) {
            L.t2 = zk;
          }
        }
      }
    }
    L.thr2 = wave_max(L.t2);
  }

  // Rank of y: a vector wholly before y counts z >= z_y (z > next_below(z_y)),
  // any other vector counts z > z_y; ties before y inside y's own vector are
  // added once when the row is finalised. Ballot totals are wave-wide.
  if (__any(cmax > cx.thr_lo)) {
    uint32_t c = 0;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int64_t last = cx.h + (i + u * BLOCK) * VEC + (VEC - 1);
      const float thr = (last < cx.y) ? cx.thr_before : cx.zy;
#pragma unroll
      for (int k = 0; k < VEC; ++k) c += __popcll(__ballot(z[u * VEC + k] > thr));
    }
    if (__lane_id() == 0) L.cnt += c;
  }

  // Sum of 2^x and of 2^x * x. A masked logit (-inf) has x = -inf and
  // 2^x = 0; x is clamped to a finite value so that 0 * x stays 0.
  const float na = -L.a;
#pragma unroll
  for (int k = 0; k < NV * VEC; k += 2) {
    const float x0 = fmaf(z[k], cx.c, na);
    const float x1 = fmaf(z[k + 1], cx.c, na);
    const float e0 = fast_exp2(x0);
    const float e1 = fast_exp2(x1);
    L.S0 += e0;
    L.S1 += e1;
    L.E0 = fmaf(e0, fmaxf(x0, -kBig), L.E0);
    L.E1 = fmaf(e1, fmaxf(x1, -kBig), L.E1);
  }
}

// One element outside the aligned vectors (row head or tail), per lane.
__device__ __forceinline__ void consume_scalar(float z, int64_t idx, const RowCtx& cx, Lane& L) {
  if (z > L.mw) lane_rescale(L, z, cx.c);
  if (z > L.t1) {
    L.t2 = L.t1;
    L.t1 = z;
    L.t1i = static_cast<int32_t>(idx);
  } else if (z > L.t2) {
    L.t2 = z;
  }
  if (cx.y >= 0) L.cnt += (z > cx.zy || (z == cx.zy && idx < cx.y)) ? 1u : 0u;
  const float x = fmaf(z, cx.c, -L.a);
  const float e = fast_exp2(x);
  L.S0 += e;
  L.E0 = fmaf(e, fmaxf(x, -kBig), L.E0);
}

// Block-wide merge of the lanes into one Partial (valid in thread 0).
template <int BLOCK>
__device__ Partial block_merge(Lane& L, float c) {
  constexpr int NW = BLOCK / kWave;
  __shared__ float sh_m[NW], sh_S[NW], sh_E[NW], sh_t1[NW], sh_t2[NW];
  __shared__ int32_t sh_t1i[NW];
  __shared__ uint32_t sh_cnt[NW];
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;

  const float mw = wave_max(L.t1);
  const uint32_t cw = wave_sum_u(L.cnt);
  float t1 = L.t1, t2 = L.t2;
  int32_t t1i = L.t1i;
  wave_top2(t1, t1i, t2);
  if (lane == 0) {
    sh_m[w] = mw;
    sh_t1[w] = t1;
    sh_t1i[w] = t1i;
    sh_t2[w] = t2;
    sh_cnt[w] = cw;
  }
  __syncthreads();
  float M = sh_m[0];
#pragma unroll
  for (int k = 1; k < NW; ++k) M = fmaxf(M, sh_m[k]);
  const float A = M * c;
  float S = L.S0 + L.S1, E = L.E0 + L.E1;
  rebase(L.a == kNegSentinel, L.a, A, S, E);
  S = wave_sum(S);
  E = wave_sum(E);
  if (lane == 0) {
    sh_S[w] = S;
    sh_E[w] = E;
  }
  __syncthreads();
  Partial p;
  p.m = M;
  p.S = 0.0f;
  p.E = 0.0f;
  p.t1 = -INFINITY;
  p.t1i = kNoIndex;
  p.t2 = -INFINITY;
  p.cnt = 0;
  p.pad = 0;
  if (threadIdx.x == 0) {
    for (int k = 0; k < NW; ++k) {
      p.S += sh_S[k];
      p.E += sh_E[k];
      top2_merge(p.t1, p.t1i, p.t2, sh_t1[k], sh_t1i[k], sh_t2[k]);
      p.cnt += sh_cnt[k];
    }
  }
  return p;
}

// Merge of G per-workgroup partial states of one row, in index order.
__device__ Partial merge_partials(const Partial* parts, int G, float c) {
  float M = parts[0].m;
  for (int g = 1; g < G; ++g) M = fmaxf(M, parts[g].m);
  const float A = M * c;
  Partial p;
  p.m = M;
  p.S = 0.0f;
  p.E = 0.0f;
  p.t1 = -INFINITY;
  p.t1i = kNoIndex;
  p.t2 = -INFINITY;
  p.cnt = 0;
  p.pad = 0;
  for (int g = 0; g < G; ++g) {
    Partial q = parts[g];
    rebase(q.m == -INFINITY, q.m * c, A, q.S, q.E);
    p.S += q.S;
    p.E += q.E;
    top2_merge(p.t1, p.t1i, p.t2, q.t1, q.t1i, q.t2);
    p.cnt += q.cnt;
  }
  return p;
}

template <typename Tin>
__device__ __forceinline__ int64_t head_elems(const void* row, int32_t V) {
  const uintptr_t addr = reinterpret_cast<uintptr_t>(row);
  const int64_t h = static_cast<int64_t>(((16u - (addr & 15u)) & 15u) / sizeof(Tin));
  return h < V ? h : V;
}

template <typename Tin>
__device__ RowCtx row_ctx(const RowArgs& a, int64_t r, const void* row) {
  RowCtx cx;
  const float T = a.temperature[r];
  // A rejected temperature still gets a finite scale, so that the
  // non-finite-logit check does not depend on it.
  cx.c = temperature_ok(T) ? kLog2e / T : kLog2e;
  cx.h = head_elems<Tin>(row, a.V);
  const int32_t y = a.sampled_ids[r];
  if (y >= 0 && y < a.V) {
    cx.y = y;
    cx.zy = Elem<Tin>::load1(row, y);
    cx.thr_before = (cx.zy == -INFINITY) ? -INFINITY : next_below(cx.zy);
    cx.thr_lo = cx.thr_before;
  } else {
    cx.y = -1;
    cx.zy = __uint_as_float(0x7fc00000u);
    cx.thr_before = INFINITY;
    cx.thr_lo = INFINITY;
  }
  return cx;
}

// Logits are read exactly once: nontemporal loads do not keep them cached.
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
#ifndef PR_CACHED_LOADS
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
#else
  return *p;
#endif
}

// Scan of the vector index range [vb, ve) of one row by one workgroup,
// plus the scalar head (first) / tail (last) elements.
// All-(-inf) vector: padding for lanes past the end of a stretch.
template <typename Tin>
__device__ __forceinline__ uint4 neg_inf_vec() {
  const uint32_t w = sizeof(Tin) == 2 ? 0xff80ff80u : 0xff800000u;
  return make_uint4(w, w, w, w);
}

// Scan of the vector index range [vb, ve) of one row by one workgroup,
// plus the scalar head (first) / tail (last) elements. Loop trip counts are
// uniform across each wave: full steps while the wave's last lane still has
// U vectors, then single-vector steps in which lanes past the end see -inf
// (a token of probability 0 that changes no result).
template <typename Tin, int BLOCK, int U>
__device__ void scan_stretch(const void* row, int32_t V, int64_t vb, int64_t ve, bool do_head, bool do_tail,
                             int64_t nvec, const RowCtx& cx, Lane& L) {
  constexpr int VEC = Elem<Tin>::kVec;
  const Tin* base = static_cast<const Tin*>(row) + cx.h;
  const uint4* vp = reinterpret_cast<const uint4*>(base);
  const int t = threadIdx.x;
  const int wave_first = t - static_cast<int>(__lane_id());
  if (do_head) {
    if (t < cx.h) consume_scalar(Elem<Tin>::load1(row, t), t, cx, L);
    const float m = wave_max(L.mw);  // one reference for the whole wave again
    if (m > L.mw) lane_rescale(L, m, cx.c);
  }
  int64_t i = vb + t;
  int64_t i_last = vb + wave_first + (kWave - 1);  // the wave's last lane
  for (; i_last + (U - 1) * BLOCK < ve; i += U * BLOCK, i_last += U * BLOCK) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = load_stream(vp + i + u * BLOCK);
    consume<Tin, U, BLOCK>(v, i, cx, L);
  }
  for (int64_t i_first = i - __lane_id(); i_first < ve; i += BLOCK, i_first += BLOCK) {
    uint4 v[1];
    v[0] = i < ve ? load_stream(vp + i) : neg_inf_vec<Tin>();
    consume<Tin, 1, BLOCK>(v, i, cx, L);
  }
  if (do_tail) {
    const int64_t tail0 = cx.h + nvec * VEC;
    for (int64_t e = tail0 + t; e < V; e += BLOCK) consume_scalar(Elem<Tin>::load1(row, e), e, cx, L);
  }
}

// Rank corrections that the vector loop leaves out, summed over the block:
// ties z == z_y before y inside y's own vector, and -- only when z_y = -inf --
// the -inf logits of the vectors before y's vector.
template <typename Tin, int BLOCK>
__device__ uint32_t rank_fixup(const void* row, int32_t V, int64_t nvec, const RowCtx& cx) {
  constexpr int VEC = Elem<Tin>::kVec;
  __shared__ uint32_t sh_fix[BLOCK / kWave];
  if (cx.y < 0) return 0;
  const int64_t vend = cx.h + nvec * VEC;
  const bool y_in_vec = cx.y >= cx.h && cx.y < vend;
  const int64_t vs = y_in_vec ? cx.h + ((cx.y - cx.h) / VEC) * VEC : 0;
  uint32_t fix = 0;
  if (y_in_vec && threadIdx.x < cx.y - vs)
    fix += (Elem<Tin>::load1(row, vs + threadIdx.x) == cx.zy) ? 1u : 0u;
  if (cx.zy == -INFINITY) {
    const int64_t lim = y_in_vec ? vs : (cx.y >= vend ? vend : cx.h);
    for (int64_t e = cx.h + threadIdx.x; e < lim; e += BLOCK)
      fix += (Elem<Tin>::load1(row, e) == -INFINITY) ? 1u : 0u;
  }
  fix = wave_sum_u(fix);
  if (threadIdx.x % kWave == 0) sh_fix[threadIdx.x / kWave] = fix;
  __syncthreads();
  uint32_t tot = 0;
  for (int k = 0; k < BLOCK / kWave; ++k) tot += sh_fix[k];
  return tot;
}

// Turns a row's merged state into the outputs (thread 0 writes). Returns the
// confidence tuple A = (logprob, maxprob, -entropy, margin) in `conf`.
__device__ void finalize_row(const RowArgs& a, int64_t r, const Partial& p, const RowCtx& cx, uint32_t fix,
                             float* conf) {
  const float T = a.temperature[r];
  uint32_t flags = 0;
  if (!temperature_ok(T)) flags |= PR_FLAG_BAD_TP;
  const bool nonfinite = !(fabsf(p.S) < INFINITY) || p.m == INFINITY || p.m == -INFINITY;
  if (nonfinite) flags |= PR_FLAG_NONFINITE;
  if (!flags && fabsf(p.m) > ldexpf(T, 100)) flags |= PR_FLAG_BAD_TP;
  if (a.top_p) {
    const float P = a.top_p[r];
    if (!(P > 0.0f)) flags |= PR_FLAG_BAD_TP;
  }
  const float qnan = __uint_as_float(0x7fc00000u);
  float max_logit = qnan, lse = qnan, entropy = qnan, logprob = qnan, maxprob = qnan, margin = qnan;
  int32_t rank = -1, argmax = -1, cutoff = -1;
  if (!(flags & (PR_FLAG_NONFINITE | PR_FLAG_BAD_TP))) {
    // S and E are relative to A = round(M * c). The exact residual
    // delta = M * c - A moves them to the exact reference M * c, so that the
    // largest logit contributes exactly 2^0 (this matters for large |M| / T).
    const float A = p.m * cx.c;
    const float delta = fmaf(p.m, cx.c, -A);
    const float sc = fast_exp2(-delta);
    const float S = p.S * sc;
    const float E = sc * fmaf(-delta, p.S, p.E);
    const float lnS = logf(S);
    max_logit = p.m / T;
    lse = max_logit + lnS;
    entropy = lnS - kLn2 * (E / S);
    maxprob = 1.0f / S;
    margin = (p.t1 - p.t2) / T;
    argmax = p.t1i;
    cutoff = a.V;
    if (cx.y >= 0) {
      rank = static_cast<int32_t>(1u + p.cnt + fix);
      const float xy = fmaf(cx.zy, cx.c, -A) - delta;
      logprob = kLn2 * xy - lnS;
    } else {
      flags |= PR_FLAG_BAD_ID;
    }
  } else if (cx.y < 0) {
    flags |= PR_FLAG_BAD_ID;
  }
  conf[0] = logprob;
  conf[1] = maxprob;
  conf[2] = -entropy;
  conf[3] = margin;
  if (a.out.max_logit) {
    a.out.max_logit[r] = max_logit;
    a.out.lse[r] = lse;
    a.out.entropy[r] = entropy;
    a.out.logprob[r] = logprob;
    a.out.maxprob[r] = maxprob;
    a.out.margin[r] = margin;
    a.out.rank[r] = rank;
    a.out.argmax[r] = argmax;
    a.out.cutoff[r] = cutoff;
    a.out.flags[r] = flags;
  }
}

// Streaming: the row's token joins its request slot's running state.
__device__ void stream_update(const StreamDev& s, int32_t slot, const float* conf) {
  if (slot < 0 || slot >= s.max_slots) return;
  const int32_t n = s.count[slot];
  s.count[slot] = n + 1;
  uint32_t nanbits = s.nanbits[slot];
  for (int f = 0; f < 4; ++f) {
    const float v = conf[f];
    if (v != v) {
      nanbits |= 1u << f;
    } else {
      s.sum[slot * 4 + f] += static_cast<double>(v);
      s.minv[slot * 4 + f] = fminf(s.minv[slot * 4 + f], v);
    }
    if (n < s.max_len) s.hist[(static_cast<int64_t>(slot) * 4 + f) * s.max_len + n] = v;
  }
  s.nanbits[slot] = nanbits;
}

}  // namespace

// MODE 0: one workgroup per row, finalised in place.
// MODE 1: G workgroups per row write partial states to a.ws.
// MODE 2: streaming; G workgroups per row, the last to finish merges,
//         finalises and updates the request slot.
// Occupancy target: 8 waves per SIMD keep enough loads in flight.
#ifndef PR_ROW_WAVES_PER_EU
#define PR_ROW_WAVES_PER_EU 8
#endif

template <typename Tin, int BLOCK, int U, int MODE>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(PR_ROW_WAVES_PER_EU)))
void row_features_kernel(RowArgs a) {
  const int G = a.G;
  const int64_t r = blockIdx.x / G;
  const int g = blockIdx.x % G;
  if (r >= a.n_rows) return;
  constexpr int VEC = Elem<Tin>::kVec;
  const void* row = static_cast<const Tin*>(a.logits) + r * a.row_stride;
  const RowCtx cx = row_ctx<Tin>(a, r, row);
  const int64_t nvec = (a.V - cx.h) / VEC;
  const int64_t vb = nvec * g / G;
  const int64_t ve = nvec * (g + 1) / G;

  Lane L;
  lane_init(L);
  scan_stretch<Tin, BLOCK, U>(row, a.V, vb, ve, g == 0, g == G - 1, nvec, cx, L);
  Partial p = block_merge<BLOCK>(L, cx.c);

  __shared__ int sh_last;
  __shared__ Partial sh_p;
  if (MODE == 1) {
    if (threadIdx.x == 0) a.ws[r * G + g] = p;
    return;
  }
  if (MODE == 2 && G > 1) {
    if (threadIdx.x == 0) {
      a.ws[r * G + g] = p;
      __threadfence();
      const uint32_t old = atomicAdd(&a.counters[r], 1u);
      sh_last = (old == static_cast<uint32_t>(G - 1));
    }
    __syncthreads();
    if (!sh_last) return;
    __threadfence();
    if (threadIdx.x == 0) {
      sh_p = merge_partials(a.ws + r * G, G, cx.c);
      a.counters[r] = 0u;
    }
    __syncthreads();
    p = sh_p;
  }
  const uint32_t fix = rank_fixup<Tin, BLOCK>(row, a.V, nvec, cx);
  if (threadIdx.x == 0) {
    float conf[4];
    finalize_row(a, r, p, cx, fix, conf);
    if (MODE == 2) stream_update(a.st, a.slot_ids[r], conf);
  }
}

// Second kernel of MODE 1: merges each row's G partials and finalises.
template <typename Tin, int BLOCK>
__global__ __launch_bounds__(BLOCK) void row_merge_kernel(RowArgs a) {
  const int64_t r = blockIdx.x;
  if (r >= a.n_rows) return;
  constexpr int VEC = Elem<Tin>::kVec;
  const void* row = static_cast<const Tin*>(a.logits) + r * a.row_stride;
  const RowCtx cx = row_ctx<Tin>(a, r, row);
  const int64_t nvec = (a.V - cx.h) / VEC;
  const uint32_t fix = rank_fixup<Tin, BLOCK>(row, a.V, nvec, cx);
  if (threadIdx.x == 0) {
    const Partial p = merge_partials(a.ws + r * a.G, a.G, cx.c);
    float conf[4];
    finalize_row(a, r, p, cx, fix, conf);
  }
}

namespace {

#ifndef PR_ROW_BLOCK
#define PR_ROW_BLOCK 128
#endif
#ifndef PR_UNROLL_BF16
#define PR_UNROLL_BF16 2
#endif
#ifndef PR_UNROLL_F32
#define PR_UNROLL_F32 4
#endif

constexpr int kBlock = PR_ROW_BLOCK;
constexpr int kTargetBlocks = 2048;  // 8 workgroups per CU on 256 CUs
constexpr int kMaxSplit = 64;

// 16-byte vectors per lane per loop step.
template <typename Tin>
constexpr int unroll_for() {
  return Elem<Tin>::kVec == 8 ? PR_UNROLL_BF16 : PR_UNROLL_F32;
}

}  // namespace

int row_split(int64_t n_rows, int32_t V, pr_dtype dtype) {
  const int VEC = dtype == PR_BF16 ? 8 : 4;
  const int64_t nvec = V / VEC;
  if (n_rows <= 0 || n_rows >= kTargetBlocks) return 1;
  int64_t G = (kTargetBlocks + n_rows - 1) / n_rows;
  const int64_t by_work = nvec / (kBlock * 4);  // at least ~4 vectors per lane
  if (G > by_work) G = by_work;
  if (G > kMaxSplit) G = kMaxSplit;
  if (G < 1) G = 1;
  return static_cast<int>(G);
}

template <typename Tin>
static hipError_t launch_typed(const RowArgs& a, int mode, hipStream_t stream) {
  constexpr int U = unroll_for<Tin>();
  const dim3 grid(static_cast<unsigned>(a.n_rows * a.G));
  if (mode == 2) {
    row_features_kernel<Tin, kBlock, U, 2><<<grid, kBlock, 0, stream>>>(a);
  } else if (a.G == 1) {
    row_features_kernel<Tin, kBlock, U, 0><<<grid, kBlock, 0, stream>>>(a);
  } else {
    row_features_kernel<Tin, kBlock, U, 1><<<grid, kBlock, 0, stream>>>(a);
    row_merge_kernel<Tin, kWave><<<dim3(static_cast<unsigned>(a.n_rows)), kWave, 0, stream>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_row_features(const RowArgs& a, pr_dtype dtype, int mode, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  return dtype == PR_BF16 ? launch_typed<uint16_t>(a, mode, stream) : launch_typed<float>(a, mode, stream);
}

}  // namespace pr
