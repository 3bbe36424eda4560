// Per-row scan machinery shared by the row-reduction and top-p kernels:
// lane state, the streaming loop over a row, block merges and the
// finalisation of a row's outputs (internal, device code only).
#pragma once

#include "row_features.h"

namespace pr {
namespace scan {

struct Lane {
  float mw;        // running max of the wave's logits (wave-uniform in the vector loop)
  float a;         // reference of S and E: mw * c, or kNegSentinel
  float S0, S1;    // two accumulators of sum 2^x (alternating elements)
  float E0, E1;    // two accumulators of sum 2^x * x
  float t1, t2;    // largest and second largest maximum of the lane's buckets (a
                   // step's vectors form one bucket, a scalar head/tail logit one)
  int32_t t1i;     // index of t1 (lowest among ties), once known
  int32_t t1v;     // first vector index of the step where t1 was set (-1: t1i is exact)
  uint32_t cnt;    // rank counts (ballot totals are added in lane 0 only)
};

struct RowCtx {
  float T;           // temperature of the row
  float c;           // log2(e) / T
  float zy;          // logit of the sampled token (NaN when y is invalid)
  float thr_before;  // strict threshold for vectors wholly before y
  float thr_lo;      // min of the two thresholds: lazy-skip test
  int32_t y;         // sampled id, or -1 when invalid
  uint32_t fix_vec;  // logits equal to z_y before y inside y's own vector
  int64_t h;         // scalar head elements before the first aligned vector
};

__device__ __forceinline__ void lane_init(Lane& L) {
  L.mw = -INFINITY;
  L.a = kNegSentinel;
  L.S0 = L.S1 = L.E0 = L.E1 = 0.0f;
  L.t1 = -INFINITY;
  L.t2 = -INFINITY;
  L.t1i = kNoIndex;
  L.t1v = -1;
  L.cnt = 0;
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

// Per-element hook of the scan: step() is called once per step with the
// step's logits z, their 2^x (relative to the lane reference L.a, after any
// rescale), the step's largest logit and its first vector index, before the
// lane's top-2 bucket maxima take the step in; scalar() likewise once per
// scalar head/tail logit with its element index; finish() once at the end
// of the stretch, before the bucket of the lane's maximum is examined. The
// feature kernel uses none.
struct NoHook {
  template <int N>
  __device__ __forceinline__ void step(const float (&)[N], const float (&)[N], float, int64_t, const Lane&) {}
  __device__ __forceinline__ void scalar(float, float, int64_t, const Lane&) {}
  __device__ __forceinline__ void finish(const Lane&) {}
};

// Two hooks run side by side.
template <typename A, typename B>
struct HookPair {
  A a;
  B b;
  template <int N>
  __device__ __forceinline__ void step(const float (&z)[N], const float (&e)[N], float cmax, int64_t i,
                                       const Lane& L) {
    a.step(z, e, cmax, i, L);
    b.step(z, e, cmax, i, L);
  }
  __device__ __forceinline__ void scalar(float z, float e, int64_t idx, const Lane& L) {
    a.scalar(z, e, idx, L);
    b.scalar(z, e, idx, L);
  }
  __device__ __forceinline__ void finish(const Lane& L) {
    a.finish(L);
    b.finish(L);
  }
};

// NV vectors of one lane; vector u has vector index i + u * BLOCK. Every lane
// of the wave calls this together (wave-uniform control flow), so the
// cross-lane steps below see all 64 lanes. With KEEP, keep[] receives the
// step's vectors whenever they raise the lane's t1 (the bucket is then read
// from registers, not memory, once the stretch is done). Without SOFT the
// sums of 2^x are not formed (a caller that takes the distribution from
// elsewhere): S0 only turns NaN on a NaN logit, so that the merged row state
// still flags it, and the hook's exps are not computed (it gets the logits).
template <typename Tin, int NV, int BLOCK, bool KEEP, bool SOFT = true, typename Hook = NoHook>
__device__ __forceinline__ void consume(const vec4u* v, int64_t i, const RowCtx& cx, Lane& L, vec4u* keep,
                                        Hook& hook) {
  constexpr int VEC = Elem<Tin>::kVec;
  float z[NV * VEC];
#pragma unroll
  for (int u = 0; u < NV; ++u) Elem<Tin>::unpack(v[u], z + u * VEC);

  float cmax = z[0];
#pragma unroll
  for (int k = 1; k < NV * VEC; ++k) cmax = fmaxf(cmax, z[k]);

  if constexpr (!SOFT) {
    bool nan = false;
#pragma unroll
    for (int k = 0; k < NV * VEC; ++k) nan |= z[k] != z[k];
    if (nan) L.S0 = __uint_as_float(0x7fc00000u);
    hook.step(z, z, cmax, i, L);
  } else {
    // The wave shares one reference, its running maximum: every exponent
    // argument stays <= 0 and the reference moves only on a new wave maximum.
    if (__any(cmax > L.mw)) lane_rescale(L, wave_max(cmax), cx.c);

    // Sum of 2^x and of 2^x * x. A masked logit (-inf) has x = -inf and
    // 2^x = 0; x is clamped to a finite value so that 0 * x stays 0.
    // The step's terms are summed on their own first and the step sums then
    // join the lane's sums: a lane that holds a term near 1 (the row's
    // maximum) would otherwise round away every term below 2^-24 added after
    // it, which in a near one-hot row (a spike 20 nats above the rest) is
    // most of S - 1 and makes log-prob err by 1e-5.
    const float na = -L.a;
    float ev[NV * VEC];
    float s0 = 0.0f, s1 = 0.0f, q0 = 0.0f, q1 = 0.0f;
#pragma unroll
    for (int k = 0; k < NV * VEC; k += 2) {
      const float x0 = fmaf(z[k], cx.c, na);
      const float x1 = fmaf(z[k + 1], cx.c, na);
      const float e0 = fast_exp2(x0);
      const float e1 = fast_exp2(x1);
      ev[k] = e0;
      ev[k + 1] = e1;
      if (k == 0) {
        s0 = e0;
        s1 = e1;
        q0 = e0 * fmaxf(x0, -kBig);
        q1 = e1 * fmaxf(x1, -kBig);
      } else {
        s0 += e0;
        s1 += e1;
        q0 = fmaf(e0, fmaxf(x0, -kBig), q0);
        q1 = fmaf(e1, fmaxf(x1, -kBig), q1);
      }
    }
    L.S0 += s0;
    L.S1 += s1;
    L.E0 += q0;
    L.E1 += q1;
    hook.step(z, ev, cmax, i, L);
  }

  // Rank of y: a vector wholly before y counts z >= z_y (z > next_below(z_y)),
  // any other vector counts z > z_y; ties before y inside y's own vector are
  // added once when the row is finalised. Ballot totals are wave-wide. (After
  // the sums, so that the first step need not wait for z_y.)
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

  // Top-1/top-2 values, per bucket: the lane keeps the largest and second
  // largest bucket maxima and the step where the largest first appeared.
  // The second value of the stretch is the larger of the second largest
  // bucket maximum and the second value inside the bucket of the maximum,
  // which is examined once the stretch is done (scan_stretch).
  const bool up = cmax > L.t1;
  L.t2 = __builtin_amdgcn_fmed3f(L.t1, L.t2, cmax);
  L.t1v = up ? static_cast<int32_t>(i) : L.t1v;
  L.t1 = fmaxf(L.t1, cmax);
  if (KEEP) {
#pragma unroll
    for (int u = 0; u < NV; ++u) keep[u] = up ? v[u] : keep[u];
  }
}

// One element outside the aligned vectors (row head or tail), per lane.
template <bool SOFT = true, typename Hook = NoHook>
__device__ __forceinline__ void consume_scalar(float z, int64_t idx, const RowCtx& cx, Lane& L, Hook& hook) {
  if (cx.y >= 0) L.cnt += (z > cx.zy || (z == cx.zy && idx < cx.y)) ? 1u : 0u;
  if constexpr (SOFT) {
    if (z > L.mw) lane_rescale(L, z, cx.c);
    const float x = fmaf(z, cx.c, -L.a);
    const float e = fast_exp2(x);
    L.S0 += e;
    L.E0 = fmaf(e, fmaxf(x, -kBig), L.E0);
    hook.scalar(z, e, idx, L);
  } else {
    if (z != z) L.S0 = __uint_as_float(0x7fc00000u);
    hook.scalar(z, z, idx, L);
  }
  // A scalar logit is a bucket of its own (t1v = -1: t1i is exact).
  if (z > L.t1) {
    L.t2 = L.t1;
    L.t1 = z;
    L.t1i = static_cast<int32_t>(idx);
    L.t1v = -1;
  } else if (z > L.t2) {
    L.t2 = z;
  }
}

// Block-wide merge of the lanes into one Partial (valid in thread 0). Each
// wave reduces its lanes to a state relative to its own largest logit and
// publishes it; after one barrier the first wave merges the NW wave states
// with lane-parallel reductions.
template <int BLOCK>
__device__ __forceinline__ Partial block_merge(Lane& L, float c) {
  constexpr int NW = BLOCK / kWave;
  static_assert(NW >= 1 && NW <= kWave, "one wave merges the wave states");
  __shared__ Partial sh[NW];
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;

  Partial q;
  q.m = wave_max(L.t1);
  float S = L.S0 + L.S1, E = L.E0 + L.E1;
  rebase(L.a == kNegSentinel, L.a, q.m * c, S, E);
  q.S = wave_sum(S);
  q.E = wave_sum(E);
  q.t1 = L.t1;
  q.t1i = L.t1i;
  q.t2 = L.t2;
  wave_top2(q.t1, q.t1i, q.t2);
  q.cnt = wave_sum_u(L.cnt);
  q.pad = 0;
  if (NW == 1) return q;
  if (lane == 0) sh[w] = q;
  __syncthreads();
  Partial p = q;
  if (w == 0) {
    Partial e;
    if (lane < NW) {
      e = sh[lane];
    } else {
      e.m = -INFINITY;
      e.S = 0.0f;
      e.E = 0.0f;
      e.t1 = -INFINITY;
      e.t1i = kNoIndex;
      e.t2 = -INFINITY;
      e.cnt = 0;
      e.pad = 0;
    }
    p.m = wave_max(e.m);
    rebase(e.m == -INFINITY, e.m * c, p.m * c, e.S, e.E);
    p.S = wave_sum(e.S);
    p.E = wave_sum(e.E);
    wave_top2(e.t1, e.t1i, e.t2);
    p.t1 = e.t1;
    p.t1i = e.t1i;
    p.t2 = e.t2;
    p.cnt = wave_sum_u(e.cnt);
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
__device__ __forceinline__ RowCtx row_ctx(const RowArgs& a, int64_t r, const void* row) {
  constexpr int VEC = Elem<Tin>::kVec;
  RowCtx cx;
  const float T = a.temperature[r];
  cx.T = T;
  // A rejected temperature still gets a finite scale, so that the
  // non-finite-logit check does not depend on it.
  cx.c = temperature_ok(T) ? kLog2e / T : kLog2e;
  cx.h = head_elems<Tin>(row, a.V);
  cx.fix_vec = 0;
  const int32_t y = a.sampled_ids ? a.sampled_ids[r] : -1;  // none yet when the kernel draws it
  if (y >= 0 && y < a.V) {
    cx.y = y;
    const int64_t q = static_cast<int64_t>(y) - cx.h;
    if (q >= 0 && q / VEC < (a.V - cx.h) / VEC) {
      // y lies in an aligned vector: one 16-byte load gives z_y and the
      // ties before y inside that vector (which the vector loop leaves out).
      const vec4u* vp = reinterpret_cast<const vec4u*>(static_cast<const Tin*>(row) + cx.h);
      float z[VEC];
      Elem<Tin>::unpack(vp[q / VEC], z);
      const int k = static_cast<int>(q % VEC);
      float zy = z[0];
#pragma unroll
      for (int j = 1; j < VEC; ++j) zy = (j == k) ? z[j] : zy;
      uint32_t f = 0;
#pragma unroll
      for (int j = 0; j < VEC - 1; ++j) f += (j < k && z[j] == zy) ? 1u : 0u;
      cx.zy = zy;
      cx.fix_vec = f;
    } else {
      cx.zy = Elem<Tin>::load1(row, y);
    }
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
__device__ __forceinline__ vec4u load_stream(const vec4u* p) {
#ifndef PR_CACHED_LOADS
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

// All-(-inf) vector: padding for lanes past the end of a stretch.
template <typename Tin>
__device__ __forceinline__ vec4u neg_inf_vec() {
  const uint32_t w = sizeof(Tin) == 2 ? 0xff80ff80u : 0xff800000u;
  return vec4u{w, w, w, w};
}

// Vector index of the first lane of the calling wave, as a wave-uniform
// (scalar) value, so that loops bounded by it compile to scalar branches.
__device__ __forceinline__ int wave_first_thread() {
  return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x));
}

// Whether every lane of the wave has LD vectors in [vb, ve).
template <int BLOCK, int LD>
__device__ __forceinline__ bool stretch_full(int64_t vb, int64_t ve) {
  return vb + wave_first_thread() + (kWave - 1) + (LD - 1) * BLOCK < ve;
}

// The first LD vectors of a lane in the vector index range [vb, ve) of a
// row (-inf past the end). Issued before the row's other inputs are read,
// so that their latency overlaps.
template <typename Tin, int BLOCK, int LD>
__device__ __forceinline__ void stretch_prefetch(const void* row, int64_t h, int64_t vb, int64_t ve, vec4u (&v)[LD]) {
  const vec4u* vp = reinterpret_cast<const vec4u*>(static_cast<const Tin*>(row) + h);
  const int64_t i = vb + threadIdx.x;
  if (stretch_full<BLOCK, LD>(vb, ve)) {
#pragma unroll
    for (int u = 0; u < LD; ++u) v[u] = load_stream(vp + i + u * BLOCK);
  } else {
#pragma unroll
    for (int u = 0; u < LD; ++u) {
      const int64_t j = i + u * BLOCK;
      v[u] = j < ve ? load_stream(vp + j) : neg_inf_vec<Tin>();
    }
  }
}

// The loop over the vector index range [vb, ve) of a row shared by every
// pass: v holds the lane's first LD vectors (stretch_prefetch); body(vv, j)
// reduces the U vectors vv[0..U) of indices j + u * BLOCK. Each lane keeps LD
// 16-byte loads in flight with two buffers: v (carried from one round to
// the next) and w (local to the round); the loads of one are issued before
// the other is reduced, so at least LD loads per lane are in flight. Loop
// trip counts are uniform across each wave: unpredicated rounds while every
// load of the round lies inside the range for the whole wave, then rounds
// whose loads are predicated, in which lanes past the end see -inf (a token
// of probability 0 that changes no result). A wave with fewer than LD
// vectors in some lane holds its whole share after the prefetch. Steps of a
// wave are reduced in increasing index order.
template <typename Tin, int BLOCK, int U, int LD, typename Body>
__device__ __forceinline__ void stream_stretch(const vec4u* vp, int64_t vb, int64_t ve, vec4u (&v)[LD], Body&& body) {
  static_assert(LD % U == 0, "load depth must be a multiple of the compute width");
  int64_t i = vb + threadIdx.x;                 // the lane's vector in v[0]
  int64_t i0 = vb + wave_first_thread();        // the same for the wave's first lane (scalar)
  if (stretch_full<BLOCK, LD>(vb, ve)) {
    for (; i0 + (kWave - 1) + (3 * LD - 1) * BLOCK < ve; i += 2 * LD * BLOCK, i0 += 2 * LD * BLOCK) {
      vec4u w[LD];
#pragma unroll
      for (int u = 0; u < LD; ++u) w[u] = load_stream(vp + i + (LD + u) * BLOCK);
#pragma unroll
      for (int c = 0; c < LD; c += U) body(v + c, i + c * BLOCK);
#pragma unroll
      for (int u = 0; u < LD; ++u) v[u] = load_stream(vp + i + (2 * LD + u) * BLOCK);
#pragma unroll
      for (int c = 0; c < LD; c += U) body(w + c, i + (LD + c) * BLOCK);
    }
    // v is inside the range; the vectors after it (fewer than 2 * LD per
    // lane) follow in at most two predicated rounds.
    for (; i0 < ve; i += LD * BLOCK, i0 += LD * BLOCK) {
      vec4u w[LD];
#pragma unroll
      for (int u = 0; u < LD; ++u) {
        const int64_t j = i + (LD + u) * BLOCK;
        w[u] = j < ve ? load_stream(vp + j) : neg_inf_vec<Tin>();
      }
#pragma unroll
      for (int c = 0; c < LD; c += U) body(v + c, i + c * BLOCK);
#pragma unroll
      for (int u = 0; u < LD; ++u) v[u] = w[u];
    }
  } else if (i0 < ve) {
#pragma unroll
    for (int c = 0; c < LD; c += U) body(v + c, i + c * BLOCK);
  }
}

// Scan of the vector index range [vb, ve) of one row by one workgroup,
// plus the scalar head (first) / tail (last) elements (stream_stretch does
// the vectors; v holds the lane's first LD vectors). SOFT as in consume().
template <typename Tin, int BLOCK, int U, int LD, bool KEEP = false, bool SOFT = true, typename Hook = NoHook>
__device__ void scan_stretch(const void* row, int32_t V, int64_t vb, int64_t ve, bool do_head, bool do_tail,
                             int64_t nvec, const RowCtx& cx, Lane& L, vec4u (&v)[LD], Hook&& hook = Hook()) {
  constexpr int VEC = Elem<Tin>::kVec;
  const Tin* base = static_cast<const Tin*>(row) + cx.h;
  const vec4u* vp = reinterpret_cast<const vec4u*>(base);
  const int t = threadIdx.x;
  vec4u keep[U];
  if (KEEP) {
#pragma unroll
    for (int u = 0; u < U; ++u) keep[u] = neg_inf_vec<Tin>();
  }
  if (do_head) {
    if (t < cx.h) consume_scalar<SOFT>(Elem<Tin>::load1(row, t), t, cx, L, hook);
    if constexpr (SOFT) {
      const float m = wave_max(L.mw);  // one reference for the whole wave again
      if (m > L.mw) lane_rescale(L, m, cx.c);
    }
  }
  stream_stretch<Tin, BLOCK, U, LD>(vp, vb, ve, v, [&](const vec4u* vv, int64_t j) {
    consume<Tin, U, BLOCK, KEEP, SOFT>(vv, j, cx, L, keep, hook);
  });
  if (do_tail) {
    const int64_t tail0 = cx.h + nvec * VEC;
    for (int64_t e = tail0 + t; e < V; e += BLOCK) consume_scalar<SOFT>(Elem<Tin>::load1(row, e), e, cx, L, hook);
  }
  hook.finish(L);
  // The lanes holding the wave maximum examine the bucket where their t1 was
  // set (kept in registers, or re-read: a few bytes per wave): its first
  // occurrence gives the exact index (ties across lanes and waves resolve by
  // index in the merges), and its other logits the second value inside it.
  const float mw = wave_max(L.t1);
  if (L.t1 == mw && L.t1v >= 0) {
    int32_t best = kNoIndex;
    uint32_t n_max = 0;
    float below = -INFINITY;
    for (int u = 0; u < U; ++u) {
      const int64_t j = static_cast<int64_t>(L.t1v) + u * BLOCK;
      if (j >= ve) break;
      float z[VEC];
      Elem<Tin>::unpack(KEEP ? keep[u] : vp[j], z);
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        if (z[k] == mw) {
          if (n_max == 0) best = static_cast<int32_t>(cx.h + j * VEC + k);
          ++n_max;
        } else {
          below = fmaxf(below, z[k]);
        }
      }
    }
    L.t1i = best;
    L.t2 = fmaxf(L.t2, n_max >= 2 ? mw : below);
  }
}

// Rank corrections that the vector loop leaves out: ties z == z_y before y
// inside y's own vector (counted when the row context was read) and -- only
// when z_y = -inf -- the -inf logits of the vectors before y's vector,
// summed over the block. z_y is the same in every thread, so the barrier
// below is reached by all threads or by none.
template <typename Tin, int BLOCK>
__device__ __forceinline__ uint32_t rank_fixup(const void* row, int32_t V, int64_t nvec, const RowCtx& cx) {
  constexpr int VEC = Elem<Tin>::kVec;
  if (cx.y < 0) return 0;
  if (cx.zy != -INFINITY) return cx.fix_vec;
  __shared__ uint32_t sh_fix[BLOCK / kWave];
  const int64_t vend = cx.h + nvec * VEC;
  const bool y_in_vec = cx.y >= cx.h && cx.y < vend;
  const int64_t vs = y_in_vec ? cx.h + ((cx.y - cx.h) / VEC) * VEC : 0;
  const int64_t lim = y_in_vec ? vs : (cx.y >= vend ? vend : cx.h);
  uint32_t fix = 0;
  for (int64_t e = cx.h + threadIdx.x; e < lim; e += BLOCK)
    fix += (Elem<Tin>::load1(row, e) == -INFINITY) ? 1u : 0u;
  fix = wave_sum_u(fix);
  if (threadIdx.x % kWave == 0) sh_fix[threadIdx.x / kWave] = fix;
  __syncthreads();
  uint32_t tot = cx.fix_vec;
  for (int k = 0; k < BLOCK / kWave; ++k) tot += sh_fix[k];
  return tot;
}

// The top-p nucleus of a row: its size k and, relative to the largest
// logit M (whose mass is 1), S = sum over the nucleus of e_v and
// E = sum over the nucleus of e_v * (z_v - M) / T, e_v = exp((z_v - M) / T).
struct Nucleus {
  int32_t k;
  double S;
  double E;
};

// Row flags known after the first pass (everything but the id and nucleus).
__device__ __forceinline__ uint32_t row_flags(const RowArgs& a, int64_t r, const Partial& p, float T) {
  uint32_t flags = 0;
  if (!temperature_ok(T)) flags |= PR_FLAG_BAD_TP;
  const bool nonfinite = !(fabsf(p.S) < INFINITY) || p.m == INFINITY || p.m == -INFINITY;
  if (nonfinite) flags |= PR_FLAG_NONFINITE;
  if (!flags && fabsf(p.m) > ldexpf(T, 100)) flags |= PR_FLAG_BAD_TP;
  if (a.top_p) {
    const float P = a.top_p[r];
    if (!(P > 0.0f)) flags |= PR_FLAG_BAD_TP;
  }
  return flags;
}

// Turns a row's merged state into the outputs (thread 0 writes). With a
// nucleus, the distribution features are those of the renormalised nucleus.
// Fills the confidence tuple A = (logprob, maxprob, -entropy, margin) and
// returns the row's flags.
__device__ __forceinline__ uint32_t finalize_row(const RowArgs& a, int64_t r, const Partial& p, const RowCtx& cx, uint32_t fix,
                                 float* conf, const Nucleus* nuc = nullptr) {
  const float T = cx.T;
  uint32_t flags = row_flags(a, r, p, T);
  const float qnan = __uint_as_float(0x7fc00000u);
  float max_logit = qnan, lse = qnan, entropy = qnan, logprob = qnan, maxprob = qnan, margin = qnan;
  int32_t rank = -1, argmax = -1, cutoff = -1;
  if (!(flags & (PR_FLAG_NONFINITE | PR_FLAG_BAD_TP))) {
    max_logit = p.m / T;
    margin = (p.t1 - p.t2) / T;
    argmax = p.t1i;
    if (cx.y >= 0) rank = static_cast<int32_t>(1u + p.cnt + fix);
    if (nuc) {
      const double lnS = ln_sum(nuc->S);
      lse = static_cast<float>(static_cast<double>(p.m) / static_cast<double>(T) + lnS);
      entropy = static_cast<float>(lnS - nuc->E / nuc->S);
      maxprob = static_cast<float>(1.0 / nuc->S);
      cutoff = nuc->k;
      if (cx.y >= 0) {
        if (rank <= nuc->k) {
          const double dy = (static_cast<double>(cx.zy) - static_cast<double>(p.m)) / static_cast<double>(T);
          logprob = static_cast<float>(dy - lnS);
        } else {
          logprob = -INFINITY;
          flags |= PR_FLAG_OUTSIDE_NUCLEUS;
        }
      }
    } else {
      // S and E are relative to A = round(M * c). The exact residual
      // delta = M * c - A moves them to the exact reference M * c, so that
      // the largest logit contributes exactly 2^0 (matters for large |M|/T).
      const float A = p.m * cx.c;
      const float delta = fmaf(p.m, cx.c, -A);
      const float sc = fast_exp2(-delta);
      const float S = p.S * sc;
      const float E = sc * fmaf(-delta, p.S, p.E);
      const float lnS = ln_sum(S);
      lse = max_logit + lnS;
      entropy = lnS - kLn2 * (E / S);
      maxprob = 1.0f / S;
      cutoff = a.V;
      if (cx.y >= 0) {
        const float xy = fmaf(cx.zy, cx.c, -A) - delta;
        logprob = kLn2 * xy - lnS;
      }
    }
  }
  if (cx.y < 0) flags |= PR_FLAG_BAD_ID;
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
  return flags;
}

// Writes row r of the verifier input sequence X: (l, m, h, rho) =
// (logprob, maxprob, -H^{top-K}, t / T) (Sec. 3.1, Eq. 3). A row whose
// distribution is undefined (non-finite logits, bad temperature or top-p)
// gets NaN in l, m and h; rho does not depend on the logits.
__device__ __forceinline__ void write_sequence_row(const RowArgs& a, int64_t r, const float* conf, uint32_t flags,
                                                   float H, float rho) {
  const bool undefined = (flags & (PR_FLAG_NONFINITE | PR_FLAG_BAD_TP)) != 0;
  float* x = a.X + r * 4;
  x[0] = conf[0];
  x[1] = conf[1];
  x[2] = undefined ? __uint_as_float(0x7fc00000u) : -H;
  x[3] = rho;
}

// Streaming: a request slot's running state, read when the row starts (a
// slot appears at most once per step, so nothing else changes it meanwhile).
struct SlotState {
  int32_t slot;  // -1: no streaming update
  int32_t n;
  uint32_t nanbits;
  double sum[4];
  float minv[4];
};

__device__ __forceinline__ SlotState slot_load(const RowArgs& a, int64_t r) {
  SlotState ss;
  ss.slot = -1;
  if (!a.slot_ids) return ss;
  const int32_t slot = a.slot_ids[r];
  if (slot < 0 || slot >= a.st.max_slots) return ss;
  ss.slot = slot;
  ss.n = a.st.count[slot];
  ss.nanbits = a.st.nanbits[slot];
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    ss.sum[f] = a.st.sum[slot * 4 + f];
    ss.minv[f] = a.st.minv[slot * 4 + f];
  }
  return ss;
}

// The row's token joins its request slot: count, sums and minima of the
// non-NaN values of A, NaN bits, and the token's A in the slot's history.
__device__ void stream_update(const StreamDev& s, const SlotState& ss, const float* conf) {
  if (ss.slot < 0) return;
  const int32_t slot = ss.slot;
  const int32_t n = ss.n;
  s.count[slot] = n + 1;
  uint32_t nanbits = ss.nanbits;
  for (int f = 0; f < 4; ++f) {
    const float v = conf[f];
    if (v != v) {
      nanbits |= 1u << f;
    } else {
      s.sum[slot * 4 + f] = ss.sum[f] + static_cast<double>(v);
      s.minv[slot * 4 + f] = fminf(ss.minv[f], v);
    }
    if (n < s.max_len) s.hist[(static_cast<int64_t>(slot) * 4 + f) * s.max_len + n] = v;
  }
  s.nanbits[slot] = nanbits;
}

}  // namespace scan
}  // namespace pr
