// Fused sample-and-verify: the token of each row is drawn from the row's
// decoding distribution softmax(z / T) inside the same pass that computes the
// verifier's features, so one read of the logits serves both (the verifier
// reads the distribution as a side product of decoding, Pro-Router, Sec. 3.1
// and Sec. 4.1).
//
// The draw is exact weighted sampling in three stages whose product is
// e_v / S for every token v:
//  - each lane scans its share of the row in buckets (kBucketSteps steps of
//    the scan; a scalar head or tail logit is a bucket of its own) and keeps
//    one bucket, replacing its choice by bucket b with probability
//    w_b / W_b, where w_b is the bucket's mass and W_b the lane's total
//    through b (sequential reservoir sampling of one item: bucket b stays
//    chosen with probability w_b / W_lane). The masses are the lane's own
//    running sums 2^x of the scan, so the test W_(b-1) < (1 - u) W_b costs an
//    add, a multiply and a compare per bucket;
//  - the row picks one lane with probability W_lane / S by inverse CDF
//    over the lanes' totals, one uniform per row;
//  - that lane's wave re-reads the bucket (kBucketSteps * U vectors, one per
//    lane) and picks a token of it with probability e_v / w_b, one more
//    uniform.
// The uniforms come from Threefry-2x32 with 13 rounds (Salmon, Moraes, Dror
// and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011), keyed
// by the caller's seed and offset, with the row and a per-draw tag as the
// counter: each uniform is a fixed function of (seed, offset, row, tag), so
// a row's token depends on its logits, its index and the workgroup size
// (how the row is split over lanes), never on timing.
#pragma once

#include "row_scan.h"

namespace pr {
namespace sample {

constexpr int kBucketSteps = 4;
constexpr uint32_t kTagScalar = 1u << 30;  // | element index: a head or tail logit
constexpr uint32_t kTagLane = 2u << 30;    // the row's choice of lane
constexpr uint32_t kTagPick = 3u << 30;    // the choice inside the chosen bucket
constexpr int32_t kNone = -1;

// Threefry-2x32-13: four rounds of add-rotate-xor between key injections.
__device__ __forceinline__ void threefry2x32(uint32_t c0, uint32_t c1, uint32_t k0, uint32_t k1, uint32_t& o0,
                                             uint32_t& o1) {
  constexpr int kRot[8] = {13, 15, 26, 6, 17, 29, 16, 24};
  const uint32_t ks[3] = {k0, k1, k0 ^ k1 ^ 0x1BD11BDAu};
  uint32_t x0 = c0 + ks[0];
  uint32_t x1 = c1 + ks[1];
#pragma unroll
  for (int r = 0; r < 13; ++r) {
    x0 += x1;
    x1 = __builtin_rotateleft32(x1, kRot[r % 8]);
    x1 ^= x0;
    if (r % 4 == 3) {
      const int s = (r + 1) / 4;
      x0 += ks[s % 3];
      x1 += ks[(s + 1) % 3] + static_cast<uint32_t>(s);
    }
  }
  o0 = x0;
  o1 = x1;
}

// A uniform in [0, 1) with 24 bits (exact in float32).
__device__ __forceinline__ float unit(uint32_t w) { return static_cast<float>(w >> 8) * 0x1p-24f; }

// Per-lane reservoir over the lane's buckets (a scan hook). Every mass is
// relative to the lane's reference L.a; when the reference moves up, the
// stored totals are moved with it. The key, the row and the step count are
// the same in every lane of a wave (the vector loop's trip counts are
// wave-uniform), so they stay in scalar registers.
struct Hook {
  uint32_t k0, k1;    // generator key (seed and offset)
  uint32_t row;       // counter word 0
  int32_t s;          // vector steps taken (bucket s / kBucketSteps)
  float Wb;           // lane total before the current bucket
  float Wl;           // lane total after the last element taken in
  float ar;           // reference of Wb and Wl
  int32_t bfirst;     // first vector index of the current bucket
  uint32_t spare;     // second random word of the current pair of buckets
  int32_t win;        // chosen bucket: its first vector index (>= 0), -(element + 2) for a scalar, or kNone

  __device__ __forceinline__ void init(uint32_t key0, uint32_t key1, int64_t r) {
    k0 = key0;
    k1 = key1;
    row = static_cast<uint32_t>(r);
    s = 0;
    Wb = Wl = 0.0f;
    ar = kNegSentinel;
    bfirst = 0;
    spare = 0;
    win = kNone;
  }
  __device__ __forceinline__ void rebase(const scan::Lane& L) {
    if (L.a != ar) {
      const float f = ar == kNegSentinel ? 0.0f : fast_exp2(ar - L.a);
      Wb *= f;
      Wl *= f;
      ar = L.a;
    }
  }
  // Keeps bucket b (mass Wl - Wb) with probability (Wl - Wb) / Wl. Buckets
  // 2j and 2j + 1 share one generator call (counter: row, thread << 20 | j).
  __device__ __forceinline__ void close(int32_t b) {
    uint32_t w = spare;
    if ((b & 1) == 0) {
      uint32_t o1;
      threefry2x32(row, (static_cast<uint32_t>(threadIdx.x) << 20) | static_cast<uint32_t>(b >> 1), k0, k1, w, o1);
      spare = o1;
    }
    if (Wb < (1.0f - unit(w)) * Wl) win = bfirst;
    Wb = Wl;
  }
  template <int N>
  __device__ __forceinline__ void step(const float (&)[N], const float (&)[N], float, int64_t i,
                                       const scan::Lane& L) {
    rebase(L);
    const int32_t su = __builtin_amdgcn_readfirstlane(s);
    if (su % kBucketSteps == 0) bfirst = static_cast<int32_t>(i);
    Wl = L.S0 + L.S1;
    s = su + 1;
    if ((su + 1) % kBucketSteps == 0) close(su / kBucketSteps);
  }
  // A partial bucket left by the vector loop is closed first.
  __device__ __forceinline__ void close_partial() {
    if (s % kBucketSteps != 0) {
      close(s / kBucketSteps);
      s += kBucketSteps - s % kBucketSteps;
    }
  }
  __device__ __forceinline__ void scalar(float, float, int64_t idx, const scan::Lane& L) {
    rebase(L);
    close_partial();
    Wl = L.S0 + L.S1;
    uint32_t o0, o1;
    threefry2x32(row, kTagScalar | (static_cast<uint32_t>(idx) & 0x3fffffffu), k0, k1, o0, o1);
    if (Wb < (1.0f - unit(o0)) * Wl) win = -static_cast<int32_t>(idx) - 2;
    Wb = Wl;
  }
  __device__ __forceinline__ void finish(const scan::Lane& L) {
    rebase(L);
    close_partial();
  }
};

struct Shared {
  float wtot[kWave];
  uint32_t pick, last;
  int32_t y;
  float zy;
};

// The row's token, after the scan: a lane by inverse CDF over the lanes'
// totals (relative to A = M * c), then a token of that lane's bucket.
// Every thread of the block calls this and gets the same (y, zy); y = -1
// when the row's distribution is undefined.
template <typename Tin, int BLOCK, int U>
__device__ void pick(const void* row, int64_t nvec, const scan::RowCtx& cx, const scan::Lane& L, const Hook& hk,
                     float A, bool defined, Shared& sh, int32_t& y, float& zy) {
  constexpr int VEC = Elem<Tin>::kVec;
  constexpr int NW = BLOCK / kWave;
  const int t = threadIdx.x;
  const int w = t / kWave;
  const int lane = t % kWave;
  float W = 0.0f;
  if (defined && L.a != kNegSentinel && hk.win != kNone) W = (L.S0 + L.S1) * fast_exp2(L.a - A);
  float incl = W;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const float v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  if (lane == kWave - 1) sh.wtot[w] = incl;
  if (t == 0) {
    sh.pick = 0xffffffffu;
    sh.last = 0xffffffffu;
    sh.y = -1;
    sh.zy = __uint_as_float(0x7fc00000u);
  }
  __syncthreads();
  float off = 0.0f, tot = 0.0f;
  for (int k = 0; k < NW; ++k) {
    off += k < w ? sh.wtot[k] : 0.0f;
    tot += sh.wtot[k];
  }
  incl += off;
  uint32_t o0, o1;
  threefry2x32(hk.row, kTagLane, hk.k0, hk.k1, o0, o1);
  const float target = unit(o0) * tot;
  if (W > 0.0f) {
    if (incl > target) atomicMin(&sh.pick, static_cast<uint32_t>(t));
    atomicMax(reinterpret_cast<int*>(&sh.last), t);  // rounding fallback: the last lane with mass
  }
  __syncthreads();
  uint32_t chosen = sh.pick;
  if (chosen == 0xffffffffu) chosen = sh.last;
  // The chosen lane's wave draws the token of its bucket: lane m holds the
  // bucket's vector m (one memory round trip for all of them), a wave scan
  // of the vectors' masses finds the vector where the running mass passes
  // u times the total, and that lane finds the token inside its vector.
  if (defined && chosen != 0xffffffffu && static_cast<int>(chosen) / kWave == w) {
    const int32_t win = __shfl(hk.win, static_cast<int>(chosen) % kWave);
    if (win <= -2) {
      if (lane == 0) {
        const int64_t e = -static_cast<int64_t>(win) - 2;
        sh.y = static_cast<int32_t>(e);
        sh.zy = Elem<Tin>::load1(row, e);
      }
    } else {
      constexpr int NB = kBucketSteps * U;
      static_assert(NB <= kWave, "one lane per vector of a bucket");
      const vec4u* vp = reinterpret_cast<const vec4u*>(static_cast<const Tin*>(row) + cx.h);
      const int64_t j = static_cast<int64_t>(win) + static_cast<int64_t>(lane) * BLOCK;
      const vec4u v = (lane < NB && j < nvec) ? vp[j] : scan::neg_inf_vec<Tin>();
      float z[VEC];
      Elem<Tin>::unpack(v, z);
      float ev[VEC];
      float part = 0.0f, zm = z[0];
      int km = 0;
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        ev[k] = fast_exp2(fmaf(z[k], cx.c, -A));
        part += ev[k];
        if (z[k] > zm) {
          zm = z[k];
          km = k;
        }
      }
      float run = part;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const float q = __shfl_up(run, o);
        if (lane >= o) run += q;
      }
      const float total = __shfl(run, kWave - 1);
      threefry2x32(hk.row, kTagPick, hk.k0, hk.k1, o0, o1);
      const float goal = unit(o0) * total;
      const int64_t base = cx.h + j * VEC;
      const uint64_t hit = __ballot(part > 0.0f && run > goal);
      if (total > 0.0f && hit != 0) {
        if (lane == __builtin_ctzll(hit)) {
          float acc = run - part;  // the running mass before this vector
          int kc = -1, klast = 0;
#pragma unroll
          for (int k = 0; k < VEC; ++k) {
            acc += ev[k];
            if (kc < 0 && ev[k] > 0.0f && acc > goal) kc = k;
            if (ev[k] > 0.0f) klast = k;
          }
          if (kc < 0) kc = klast;  // rounding inside the vector
          float zc = z[0];
#pragma unroll
          for (int k = 1; k < VEC; ++k) zc = k == kc ? z[k] : zc;
          sh.y = static_cast<int32_t>(base + kc);
          sh.zy = zc;
        }
      } else {  // every mass below float range: the bucket's largest logit
        const float zmax = wave_max(zm);
        const uint64_t at = __ballot(zm == zmax);
        if (lane == __builtin_ctzll(at)) {
          sh.y = static_cast<int32_t>(base + km);
          sh.zy = zm;
        }
      }
    }
  }
  __syncthreads();
  y = sh.y;
  zy = sh.zy;
}

}  // namespace sample
}  // namespace pr
