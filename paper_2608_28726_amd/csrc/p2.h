// Bounded-memory tail quantile of the streaming state: the P-square
// estimator of R. Jain and I. Chlamtac (CACM 28(10), 1985), one per slot and
// confidence column, in float64.
//
// Five markers per column track the minimum, the p/2-, p-, (1+p)/2-quantiles
// and the maximum of the column's observations. Each observation increments
// the positions of the markers above its cell; each interior marker whose
// position is at least one away from its desired position 1 + (N-1) f_i,
// f = (0, p/2, p, (1+p)/2, 1), moves one place towards it, its height
// predicted by the piecewise-parabolic formula through its two neighbours,
// or linearly towards the neighbour it moves to when the parabola leaves the
// neighbours' interval. With at most five observations the markers are the
// observations themselves and the estimate is their exact nearest-rank
// quantile. NaN is not fed; an infinite value is not fed either and marks
// the column's estimate NaN (the interpolation is undefined on infinite
// heights). The arithmetic is written in a fixed order and the library is
// built without floating-point contraction, so the same observations give
// the same heights on every run.
#pragma once

#include "row_features.h"

namespace pr {
namespace p2 {

// State of one slot: heights q_i of column f at q[(slot * 5 + i) * 4 + f];
// positions of markers 1..3 and the number of observations fed (-1 once an
// infinite value was seen) at n[(slot * 4 + j) * 4 + f]. The lowest marker's
// position is always 1 and the highest one's the number fed.
__device__ __forceinline__ double* heights(const StreamDev& s, int32_t slot, int f) {
  return s.p2q + static_cast<int64_t>(slot) * 20 + f;
}
__device__ __forceinline__ int32_t* positions(const StreamDev& s, int32_t slot, int f) {
  return s.p2n + static_cast<int64_t>(slot) * 16 + f;
}

// Stable ascending sort of five values (adjacent swaps of strictly greater
// pairs only).
__device__ __forceinline__ void sort5(double* v) {
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
#pragma unroll
    for (int j = 0; j < 4 - pass; ++j) {
      if (v[j] > v[j + 1]) {
        const double t = v[j];
        v[j] = v[j + 1];
        v[j + 1] = t;
      }
    }
  }
}

// One column's marker state as read from memory.
struct Markers {
  double q[5];
  int32_t n1, n2, n3, fed;
};

__device__ __forceinline__ Markers load(const StreamDev& s, int32_t slot, int f) {
  const int32_t* nb = positions(s, slot, f);
  const double* qb = heights(s, slot, f);
  Markers m;
#pragma unroll
  for (int i = 0; i < 5; ++i) m.q[i] = qb[4 * i];
  m.n1 = nb[0];
  m.n2 = nb[4];
  m.n3 = nb[8];
  m.fed = nb[12];
  return m;
}

// Feeds one observation of column f to the slot's markers, whose state m was
// read before (nothing else changes it meanwhile: a slot takes at most one
// token per step).
__device__ void feed(const StreamDev& s, int32_t slot, int f, float v, const Markers& m) {
  int32_t* nb = positions(s, slot, f);
  double* qb = heights(s, slot, f);
  const int32_t fed = m.fed;
  if (fed < 0 || v != v) return;
  if (__builtin_isinf(v)) {
    nb[12] = -1;
    return;
  }
  const int32_t N = fed + 1;
  nb[12] = N;
  const double x = static_cast<double>(v);
  if (N <= 5) {
    if (N < 5) {
      qb[4 * (N - 1)] = x;
      return;
    }
    double q[5] = {m.q[0], m.q[1], m.q[2], m.q[3], x};
    sort5(q);
#pragma unroll
    for (int i = 0; i < 5; ++i) qb[4 * i] = q[i];
    nb[0] = 2;
    nb[4] = 3;
    nb[8] = 4;
    return;
  }
  double q[5];
  int32_t n[5];
#pragma unroll
  for (int i = 0; i < 5; ++i) q[i] = m.q[i];
  n[0] = 1;
  n[1] = m.n1;
  n[2] = m.n2;
  n[3] = m.n3;
  n[4] = N - 1;
  // The cell k with q_k <= x < q_(k+1); the extreme markers follow the
  // extremes. The heights stay ordered, so the cell is the number of
  // interior markers at or below x.
  int k;
  if (x < q[0]) {
    q[0] = x;
    k = 0;
  } else if (x >= q[4]) {
    if (x > q[4]) q[4] = x;
    k = 3;
  } else {
    k = (x >= q[1] ? 1 : 0) + (x >= q[2] ? 1 : 0) + (x >= q[3] ? 1 : 0);
  }
#pragma unroll
  for (int i = 1; i < 5; ++i) n[i] += i > k ? 1 : 0;
  const double p = s.p2p;
  const double f_i[5] = {0.0, p / 2.0, p, (1.0 + p) / 2.0, 1.0};
#pragma unroll
  for (int i = 1; i <= 3; ++i) {
    const double d = (1.0 + static_cast<double>(N - 1) * f_i[i]) - static_cast<double>(n[i]);
    if ((d >= 1.0 && n[i + 1] - n[i] > 1) || (d <= -1.0 && n[i - 1] - n[i] < -1)) {
      const int32_t sg = d > 0.0 ? 1 : -1;
      const double sd = static_cast<double>(sg);
      double qp = q[i] + sd / static_cast<double>(n[i + 1] - n[i - 1]) *
                             (static_cast<double>(n[i] - n[i - 1] + sg) * (q[i + 1] - q[i]) /
                                  static_cast<double>(n[i + 1] - n[i]) +
                              static_cast<double>(n[i + 1] - n[i] - sg) * (q[i] - q[i - 1]) /
                                  static_cast<double>(n[i] - n[i - 1]));
      if (!(q[i - 1] < qp && qp < q[i + 1])) {
        qp = sg > 0 ? q[i] + sd * (q[i + 1] - q[i]) / static_cast<double>(n[i + 1] - n[i])
                    : q[i] + sd * (q[i - 1] - q[i]) / static_cast<double>(n[i - 1] - n[i]);
      }
      q[i] = qp;
      n[i] += sg;
    }
  }
#pragma unroll
  for (int i = 0; i < 5; ++i) qb[4 * i] = q[i];
  nb[0] = n[1];
  nb[4] = n[2];
  nb[8] = n[3];
}

// The slot of row r when its markers are to be fed (streaming in
// bounded-memory mode), else -1.
__device__ __forceinline__ int32_t row_slot(const RowArgs& a, int64_t r) {
  if (!a.slot_ids || !a.st.p2q) return -1;
  const int32_t slot = a.slot_ids[r];
  return slot >= 0 && slot < a.st.max_slots ? slot : -1;
}

// Lane f < 4 of the finalising wave reads column f's markers of row r's slot
// (early, so that the latency hides behind the row).
struct RowMarkers {
  int32_t slot;
  Markers m;
  __device__ __forceinline__ void fetch(const RowArgs& a, int64_t r) {
    slot = row_slot(a, r);
    const int lane = threadIdx.x % kWave;
    if (slot >= 0 && lane < 4) m = load(a.st, slot, lane);
  }
};

// The row's token joins its slot's markers: the confidence tuple is held by
// lane 0 of the calling wave, lanes 0..3 feed columns 0..3 from the state
// fetched before. Every lane of the wave must call this.
__device__ __forceinline__ void feed_row(const RowArgs& a, const RowMarkers& rm, const float* conf) {
  const int lane = threadIdx.x % kWave;
  float v = 0.0f;
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    const float t = __shfl(conf[f], 0);
    if (lane == f) v = t;
  }
  if (rm.slot >= 0 && lane < 4) feed(a.st, rm.slot, lane, v, rm.m);
}

// The estimate of column f: NaN when nothing was fed or an infinite value
// was seen; the exact nearest-rank quantile of j = max(1, ceil(p * N)) with
// at most five observations; the middle marker's height otherwise.
__device__ float estimate(const StreamDev& s, int32_t slot, int f) {
  const int32_t N = positions(s, slot, f)[12];
  if (N <= 0) return __uint_as_float(0x7fc00000u);
  const double* qb = heights(s, slot, f);
  if (N > 5) return static_cast<float>(qb[8]);
  double v[5];
#pragma unroll
  for (int i = 0; i < 5; ++i) v[i] = i < N ? qb[4 * i] : INFINITY;
  sort5(v);
  int64_t j = static_cast<int64_t>(ceil(s.p2p * static_cast<double>(N)));
  if (j < 1) j = 1;
  if (j > N) j = N;
  double e = v[0];
#pragma unroll
  for (int i = 1; i < 5; ++i) e = j == i + 1 ? v[i] : e;
  return static_cast<float>(e);
}

}  // namespace p2
}  // namespace pr
