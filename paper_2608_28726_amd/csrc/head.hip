// The paper's verifier head on the GPU (Pro-Router, Sec. 3.1, the paragraph
// after Eq. 3; Sec. 4.2): each request's input sequence X (T tokens x 4
// features) is projected to 64 features with a sinusoidal positional
// encoding, passes two post-norm transformer encoder layers (4 heads of 16,
// feed-forward width 128, LayerNorm eps 1e-5), is mean-pooled over its
// tokens and mapped to one shipping confidence by a linear map and a sigmoid.
//
// The tokens of all requests are processed together as rows:
//  head_qkv_kernel   64-row tiles: (first layer: projection + encoding), the
//                    QKV projection on MFMA (v_mfma_f32_16x16x4f32);
//  head_plan_kernel  one workgroup: the attention's work items (request,
//                    head, 64 queries), the heaviest first;
//  head_attn_kernel  persistent workgroups of 4 waves that take the items in
//                    that order; 16 queries per wave over all of the
//                    request's keys: scores and value products on MFMA,
//                    online softmax per query;
//  head_ffn_kernel   64-row tiles: output projection, residual, LayerNorm,
//                    feed-forward (MFMA), residual, LayerNorm;
//  head_pool_kernel  one workgroup per request: mean pool, linear, sigmoid.
// Everything is float32 with float32 accumulation.
#include "head.h"

namespace pr {

namespace {

constexpr int D = kHeadD;       // 64
constexpr int FF = kHeadFF;     // 128
constexpr int NH = kHeadHeads;  // 4
constexpr int DH = D / NH;      // 16
constexpr int QKV = 3 * D;      // 192
constexpr int kTile = 64;       // rows per tile
constexpr int kTileThreads = 256;
constexpr float kLnEps = 1e-5f;

typedef float f4 __attribute__((ext_vector_type(4)));

// Offsets (floats) of the parameter tensors in the flat weight buffer.
constexpr int kW_in = 0;
constexpr int kB_in = kW_in + D * 4;
constexpr int kLayer0 = kB_in + D;
constexpr int kLayerSize = QKV * D + QKV + D * D + D + 2 * D + FF * D + FF + D * FF + D + 2 * D;
constexpr int kW_qkv = 0, kB_qkv = kW_qkv + QKV * D, kW_o = kB_qkv + QKV, kB_o = kW_o + D * D;
constexpr int kLn1g = kB_o + D, kLn1b = kLn1g + D, kW_1 = kLn1b + D, kB_1 = kW_1 + FF * D;
constexpr int kW_2 = kB_1 + FF, kB_2 = kW_2 + D * FF, kLn2g = kB_2 + D, kLn2b = kLn2g + D;
constexpr int kW_out = kLayer0 + kHeadLayers * kLayerSize;
constexpr int kB_out = kW_out + D;
static_assert(kLayerSize == 33472 && kB_out + 1 == kHeadWeights, "parameter layout");
static_assert(kLn2b + D == kLayerSize, "layer layout");

// Padded LDS row strides (floats): rows of a tile start on different banks.
constexpr int kSA = D + 4;   // 64-wide activations and weights
constexpr int kSF = FF + 4;  // 128-wide

// Largest i with offsets[i] <= r (offsets non-decreasing, offsets[0] <= r).
__device__ int64_t request_of(const int32_t* offsets, int32_t n_req, int64_t r) {
  int64_t lo = 0, hi = n_req - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (offsets[mid] <= r) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// C (64 x 16*NB) += A (64 x K, LDS, stride sa) x B^T, B = W (16*NB rows x K,
// LDS, stride sw): wave w computes row block w; acc[j] is column block j in
// the MFMA output layout (lane l, register r: row 4*(l/16) + r, column l%16
// of the 16 x 16 block). The contraction runs in blocks of 16: product m =
// 0..3 of a block takes k = k0 + 4 (l / 16) + m in lane l (any assignment
// of a block's 16 values of k works when A and B share it), so that a lane
// reads its four values of A and of each row of B with one 16-byte LDS
// load. Rows start 16-byte aligned; their strides (68 and 132 floats) are 4
// modulo the 64 banks, so the 16 lanes of one k group read 16 distinct
// groups of 4 banks.
template <int NB, int K>
__device__ __forceinline__ void tile_gemm(const float* A, int sa, const float* W, int sw, f4 (&acc)[NB]) {
  static_assert(K % 16 == 0, "blocks of 16 along the contraction");
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;
  const int ar = 16 * w + lane % 16;
  const int kq = lane / 16;
#pragma unroll 2
  for (int k0 = 0; k0 < K; k0 += 16) {
    const f4 a4 = *reinterpret_cast<const f4*>(A + ar * sa + k0 + 4 * kq);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const f4 b4 = *reinterpret_cast<const f4*>(W + (16 * j + lane % 16) * sw + k0 + 4 * kq);
#pragma unroll
      for (int m = 0; m < 4; ++m) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[m], b4[m], acc[j], 0, 0, 0);
    }
  }
}

// Copies ROWS x COLS floats (row-major, global) into LDS with row stride S,
// as 16-byte vectors: every load of a thread is issued before its first
// store, so the copy costs one memory round trip. stage_load and
// stage_store are its halves, for a copy whose loads are issued early and
// stored once the LDS is free.
template <int ROWS, int COLS>
struct Staged {
  static constexpr int kVecs = ROWS * COLS / 4;
  static_assert(kVecs % kTileThreads == 0 && COLS % 4 == 0, "whole vectors per thread");
  f4 v[kVecs / kTileThreads];
};
template <int ROWS, int COLS>
__device__ __forceinline__ void stage_load(Staged<ROWS, COLS>& st, const float* src) {
  const f4* s4 = reinterpret_cast<const f4*>(src);
#pragma unroll
  for (int k = 0; k < Staged<ROWS, COLS>::kVecs / kTileThreads; ++k) st.v[k] = s4[threadIdx.x + k * kTileThreads];
}
template <int ROWS, int COLS, int S>
__device__ __forceinline__ void stage_store(float* dst, const Staged<ROWS, COLS>& st) {
  static_assert(S % 4 == 0, "rows of whole vectors");
#pragma unroll
  for (int k = 0; k < Staged<ROWS, COLS>::kVecs / kTileThreads; ++k) {
    const int i = threadIdx.x + k * kTileThreads;
    *reinterpret_cast<f4*>(dst + (i / (COLS / 4)) * S + (i % (COLS / 4)) * 4) = st.v[k];
  }
}
template <int ROWS, int COLS, int S>
__device__ __forceinline__ void stage(float* dst, const float* src) {
  Staged<ROWS, COLS> st;
  stage_load(st, src);
  stage_store<ROWS, COLS, S>(dst, st);
}

// The same for rows r0 .. r0+63 of a [n_rows][64] activation array (rows
// past the end read as zero).
__device__ __forceinline__ void stage_rows(float* dst, const float* src, int64_t r0, int64_t n_rows) {
  constexpr int kPer = kTile * D / 4 / kTileThreads;
  f4 v[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int i = threadIdx.x + k * kTileThreads;
    const int64_t r = r0 + i / (D / 4);
    v[k] = r < n_rows ? reinterpret_cast<const f4*>(src + r * D)[i % (D / 4)] : f4{0.0f, 0.0f, 0.0f, 0.0f};
  }
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int i = threadIdx.x + k * kTileThreads;
    *reinterpret_cast<f4*>(dst + (i / (D / 4)) * kSA + (i % (D / 4)) * 4) = v[k];
  }
}

// LayerNorm of the 64 values of each row held by the 16 lanes l / 16 = q of a
// wave (4 column blocks x 4 rows per lane, MFMA layout): x[j][r] is row
// 4q + r, column 16 j + l % 16, whose gain and bias are g[j] and b[j].
// Biased variance, eps 1e-5.
__device__ __forceinline__ void layer_norm_rows(f4 (&x)[4], const float (&g)[4], const float (&b)[4]) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float s = x[0][r] + x[1][r] + x[2][r] + x[3][r];
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) s += __shfl_xor(s, o, 16);
    const float mu = s * (1.0f / D);
    float v = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float d = x[j][r] - mu;
      v = fmaf(d, d, v);
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 16);
    const float inv = 1.0f / sqrtf(v * (1.0f / D) + kLnEps);
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j][r] = fmaf((x[j][r] - mu) * inv, g[j], b[j]);
  }
}

// A lane's values of NB consecutive 16-column blocks of a parameter vector
// (column 16 j + l % 16), loaded when a kernel starts so that their latency
// overlaps the staging.
template <int NB>
__device__ __forceinline__ void lane_cols(float (&out)[NB], const float* v) {
#pragma unroll
  for (int j = 0; j < NB; ++j) out[j] = v[16 * j + threadIdx.x % 16];
}

}  // namespace

// QKV projection of a 64-row tile; FIRST: the rows are made from X first
// (projection + positional encoding) and written to H.
template <bool FIRST>
__global__ __launch_bounds__(kTileThreads) void head_qkv_kernel(HeadArgs a, int layer, const float* Hin,
                                                               float* Hout) {
  __shared__ __attribute__((aligned(16))) float sA[kTile * kSA];
  __shared__ __attribute__((aligned(16))) float sW[QKV * kSA];
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kTile;
  const float* Wl = a.weights + kLayer0 + layer * kLayerSize;
  float bias[QKV / 16];
  lane_cols(bias, Wl + kB_qkv);
  if (FIRST) {
    // row position t - 1 within its request, one thread per row
    __shared__ int32_t sPos[kTile];
    if (threadIdx.x < kTile) {
      const int64_t r = r0 + threadIdx.x;
      int32_t pos = 0;
      if (r < a.n_rows) pos = static_cast<int32_t>(r - a.offsets[request_of(a.offsets, a.n_req, r)]);
      sPos[threadIdx.x] = pos;
    }
    __syncthreads();
    // A thread keeps one feature pair (2p, 2p + 1) of its rows: the sine and
    // the cosine of (t - 1) f_p, f_p = 10000^(-2p / 64). The angle is formed
    // and reduced to [-pi, pi] in float64 (positions reach 10^3), its sine
    // and cosine taken together in float32.
    constexpr int kPairs = D / 2;
    static_assert(kTileThreads % kPairs == 0, "a thread's pair is the same in every row");
    const int j0 = 2 * (threadIdx.x % kPairs);
    const double freq = exp2(-static_cast<double>(j0) / D * 13.287712379549449);
    const float* w0 = a.weights + kW_in + j0 * 4;
    const float* w1 = w0 + 4;
    for (int i = threadIdx.x; i < kTile * kPairs; i += kTileThreads) {
      const int rr = i / kPairs;
      const int64_t r = r0 + rr;
      float h0 = 0.0f, h1 = 0.0f;
      if (r < a.n_rows) {
        const float* x = a.X + r * 4;
        h0 = a.weights[kB_in + j0];
        h1 = a.weights[kB_in + j0 + 1];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          h0 = fmaf(w0[c], x[c], h0);
          h1 = fmaf(w1[c], x[c], h1);
        }
        const double angle = static_cast<double>(sPos[rr]) * freq;
        const double red = fma(-rint(angle * 0.15915494309189535), 6.283185307179586, angle);
        float sn, cs;
        sincosf(static_cast<float>(red), &sn, &cs);
        h0 += sn;
        h1 += cs;
        Hout[r * D + j0] = h0;
        Hout[r * D + j0 + 1] = h1;
      }
      sA[rr * kSA + j0] = h0;
      sA[rr * kSA + j0 + 1] = h1;
    }
  } else {
    stage_rows(sA, Hin, r0, a.n_rows);
  }
  stage<QKV, D, kSA>(sW, Wl + kW_qkv);
  __syncthreads();
  f4 acc[QKV / 16];
#pragma unroll
  for (int j = 0; j < QKV / 16; ++j) acc[j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
  tile_gemm<QKV / 16, D>(sA, kSA, sW, kSA, acc);
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
#pragma unroll
  for (int j = 0; j < QKV / 16; ++j) {
    const int col = 16 * j + lane % 16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = r0 + 16 * w + 4 * (lane / 16) + r;
      if (row < a.n_rows) a.qkv[row * QKV + col] = acc[j][r] + bias[j];
    }
  }
}

// Scaled dot-product attention of 64 queries of one request and one head
// over all of the request's keys, on MFMA. Each of the 4 waves takes 16
// queries; the workgroup stages the keys and values in tiles of 64 (double
// buffered in LDS, K by key and V transposed, so that a lane reads its four
// operands of a group of products with one 16-byte load; a tile's loads are
// issued before the current tile is computed and stored after).
// Per group of 16 keys a wave computes the transposed scores S^T = K Q^T
// with four v_mfma_f32_16x16x4f32 over the 16 dimensions (queries
// pre-scaled by log2(e) / sqrt(16)), so that lane l holds the scores of
// query l % 16 for keys 4 (l / 16) + r, r = 0..3. The 4 groups of a tile are
// independent chains; one online-softmax update per tile and query in base
// 2 (a query's 64 keys lie in 16 registers of 4 lanes: two cross-lane steps
// for the maximum, two for the sum); then O += P V with 16 more, taking each
// group's keys in the order 4m + r, in which the score registers already
// are the matrix A operand.
constexpr int kAttnWaves = 4;
constexpr int kAttnQ = 16;                      // queries per wave
constexpr int kAttnWgQ = kAttnWaves * kAttnQ;   // queries per workgroup
#ifndef PR_ATTN_KT
#define PR_ATTN_KT 64
#endif
constexpr int kKT = PR_ATTN_KT;                 // keys per staged tile (one softmax update)
constexpr int kKC = kKT * 4 / (kAttnWaves * kWave);  // a thread's (key, 4 dimensions) chunks of a tile
static_assert(kKC >= 1 && kKC * kAttnWaves * kWave == kKT * 4, "whole chunks per thread");
// K as rows of one key and V transposed, rows of one dimension; the padding
// keeps rows 16-byte aligned and a 16-lane group's 16-byte reads (rows 20
// or 68 floats apart, 4 banks each) free of bank conflicts
constexpr int kKPad = DH + 4;
constexpr int kVPad = kKT + 4;
#ifndef PR_ATTN_PER_CU
#define PR_ATTN_PER_CU 2
#endif
constexpr int kAttnPersist = PR_ATTN_PER_CU * 256;  // persistent attention workgroups
typedef float fx4 __attribute__((ext_vector_type(4)));

// One work item: queries [q0, q0 + 64) of request [lo, hi) and head hd. Every
// thread of the workgroup takes the same number of barriers; the LDS buffers
// are free again when it returns.
__device__ __forceinline__ void attend(const HeadArgs& a, int64_t lo, int64_t hi, int hd, int64_t q0,
                                       float (&sK)[2][kKT * kKPad], float (&sV)[2][DH * kVPad]) {
  const int64_t T = hi - lo;
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int i16 = lane % 16, g = lane / 16;
  const int64_t qw = q0 + w * kAttnQ;  // this wave's first query
  constexpr float kScale = 1.4426950408889634f / 4.0f;  // log2(e) / sqrt(DH)
  // B operand of S^T: Q[qw + i16][4g + c] for product c = 0..3 (each lane
  // group g contracts over its own four consecutive dimensions)
  float qb[4];
  {
    const int64_t q = qw + i16;
    const bool ok = q < hi;
    const f4 q4 = *reinterpret_cast<const f4*>(a.qkv + (ok ? q : lo) * QKV + hd * DH + 4 * g);
#pragma unroll
    for (int c = 0; c < 4; ++c) qb[c] = ok ? q4[c] * kScale : 0.0f;
  }
  // A thread's chunks of a tile: keys kk0 + 64 c, 4 dimensions each.
  constexpr int kKeysPerRound = kAttnWaves * kWave / 4;
  const int kk0 = threadIdx.x / 4, d4 = threadIdx.x % 4;
  auto load = [&](int64_t t, f4 (&kv)[kKC], f4 (&vv)[kKC]) {
#pragma unroll
    for (int c = 0; c < kKC; ++c) {
      const int64_t key = lo + t * kKT + kk0 + kKeysPerRound * c;
      kv[c] = f4{0.0f, 0.0f, 0.0f, 0.0f};
      vv[c] = kv[c];
      if (key < hi) {
        const f4* src = reinterpret_cast<const f4*>(a.qkv + key * QKV);
        kv[c] = src[(D + hd * DH) / 4 + d4];
        vv[c] = src[(2 * D + hd * DH) / 4 + d4];
      }
    }
  };
  auto store = [&](int buf, const f4 (&kv)[kKC], const f4 (&vv)[kKC]) {
#pragma unroll
    for (int c = 0; c < kKC; ++c) {
      const int kk = kk0 + kKeysPerRound * c;
      *reinterpret_cast<f4*>(&sK[buf][kk * kKPad + 4 * d4]) = kv[c];
#pragma unroll
      for (int e = 0; e < 4; ++e) sV[buf][(4 * d4 + e) * kVPad + kk] = vv[c][e];
    }
  };
  float m = -INFINITY, l = 0.0f;  // of query i16 (the same in its 4 lanes)
  fx4 acc = fx4{0.0f, 0.0f, 0.0f, 0.0f};  // O[4g + r][i16]
  const int64_t ntiles = (T + kKT - 1) / kKT;
  const bool busy = qw < hi;  // a wave whose queries all lie past the request only stages
  f4 nk[kKC], nv[kKC];
  load(0, nk, nv);
  store(0, nk, nv);
  __syncthreads();
  for (int64_t t = 0; t < ntiles; ++t) {
    const int buf = static_cast<int>(t & 1);
    if (t + 1 < ntiles) load(t + 1, nk, nv);
    if (busy) {
      const float* K = sK[buf];
      const float* Vs = sV[buf];
      const int64_t kt0 = lo + t * kKT;
      fx4 st[kKT / 16];
#pragma unroll
      for (int sub = 0; sub < kKT / 16; ++sub) {
        const f4 k4 = *reinterpret_cast<const f4*>(&K[(sub * 16 + i16) * kKPad + 4 * g]);
        st[sub] = fx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < 4; ++c) st[sub] = __builtin_amdgcn_mfma_f32_16x16x4f32(k4[c], qb[c], st[sub], 0, 0, 0);
      }
      float s[kKT / 4];
      float tm = -INFINITY;
#pragma unroll
      for (int sub = 0; sub < kKT / 16; ++sub) {
        const float v[4] = {st[sub].x, st[sub].y, st[sub].z, st[sub].w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool key_ok = kt0 + sub * 16 + 4 * g + r < hi;  // keys past the request: probability 0
          s[4 * sub + r] = key_ok ? v[r] : -INFINITY;
          tm = fmaxf(tm, s[4 * sub + r]);
        }
      }
      tm = fmaxf(tm, __shfl_xor(tm, 16));
      tm = fmaxf(tm, __shfl_xor(tm, 32));
      const float mn = fmaxf(m, tm);  // finite: the tile's first key is a key of the request
      const float corr = exp2f(m - mn);  // m = -inf at first: 0
      float ps = 0.0f;
#pragma unroll
      for (int k = 0; k < kKT / 4; ++k) {
        s[k] = exp2f(s[k] - mn);
        ps += s[k];
      }
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      l = fmaf(l, corr, ps);
      m = mn;
      // row 4g + r of O belongs to query 4g + r, whose factor lane 4g + r holds
      acc.x *= __shfl(corr, 4 * g);
      acc.y *= __shfl(corr, 4 * g + 1);
      acc.z *= __shfl(corr, 4 * g + 2);
      acc.w *= __shfl(corr, 4 * g + 3);
#pragma unroll
      for (int sub = 0; sub < kKT / 16; ++sub) {
        // V[sub 16 + 4g + r][i16], r = 0..3: four consecutive keys of row i16 of V^T
        const f4 v4 = *reinterpret_cast<const f4*>(&Vs[i16 * kVPad + sub * 16 + 4 * g]);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(s[4 * sub + r], v4[r], acc, 0, 0, 0);
      }
    }
    if (t + 1 < ntiles) store(buf ^ 1, nk, nv);
    __syncthreads();  // tile t + 1 is staged; buffer buf is free for tile t + 2
  }
  if (!busy) return;
  const float o[4] = {acc.x, acc.y, acc.z, acc.w};
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float lq = __shfl(l, 4 * g + r);
    const int64_t q = qw + 4 * g + r;
    if (q < hi) a.att[q * D + hd * DH + i16] = o[r] / lq;
  }
}

// Persistent: each workgroup takes work items in list order (the heaviest
// first) until the list of the layer is used up, so that workgroups that
// drew short requests take more of them. Every workgroup ends when it draws
// an index past the item count.
__global__ __launch_bounds__(kAttnWaves * kWave) void head_attn_kernel(HeadArgs a, int layer) {
  __shared__ __attribute__((aligned(16))) float sK[2][kKT * kKPad];
  __shared__ __attribute__((aligned(16))) float sV[2][DH * kVPad];
  __shared__ int32_t s_item;
  const int32_t n_items = a.ctl[0];
  for (;;) {
    if (threadIdx.x == 0) s_item = atomicAdd(&a.ctl[1 + layer], 1);
    __syncthreads();
    const int32_t it = s_item;
    __syncthreads();  // every thread has read s_item before the next draw
    if (it >= n_items) return;
    const int32_t req = a.items[2 * it];
    const int32_t ht = a.items[2 * it + 1];
    const int64_t lo = a.offsets[req], hi = a.offsets[req + 1];
    attend(a, lo, hi, ht & 3, lo + static_cast<int64_t>(ht >> 2) * kAttnWgQ, sK, sV);
  }
}

// The attention's work list: for every request of 1..max_len tokens, its
// kHeadHeads x ceil(T / 64) items (head, 64 queries), ordered by the
// request's number of key tiles, largest first (a counting sort over that
// number, clamped to kPlanBins - 1), and the counters of the two layers set
// to zero. One workgroup.
constexpr int kPlanThreads = 1024;
constexpr int kPlanBins = 1024;
__global__ __launch_bounds__(kPlanThreads) void head_plan_kernel(HeadArgs a) {
  __shared__ int32_t cnt[kPlanBins];
  __shared__ int32_t pos[kPlanBins];
  for (int b = threadIdx.x; b < kPlanBins; b += kPlanThreads) cnt[b] = 0;
  __syncthreads();
  auto tiles_of = [&](int32_t r) -> int32_t {
    const int64_t T = static_cast<int64_t>(a.offsets[r + 1]) - a.offsets[r];
    return (T >= 1 && T <= a.max_len) ? static_cast<int32_t>((T + kAttnWgQ - 1) / kAttnWgQ) : 0;
  };
  for (int32_t r = threadIdx.x; r < a.n_req; r += kPlanThreads) {
    const int32_t nt = tiles_of(r);
    if (nt > 0) atomicAdd(&cnt[nt < kPlanBins ? nt : kPlanBins - 1], NH * nt);
  }
  __syncthreads();
  {  // starting positions, largest bin first: thread j takes bin kPlanBins - 1 - j
    static_assert(kPlanBins == kPlanThreads, "one bin per thread");
    __shared__ int32_t wsum[kPlanThreads / kWave];
    const int j = threadIdx.x, lane = j % kWave, wv = j / kWave;
    const int32_t c = cnt[kPlanBins - 1 - j];
    int32_t x = c;  // inclusive scan within the wave
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const int32_t t = __shfl_up(x, d);
      if (lane >= d) x += t;
    }
    if (lane == kWave - 1) wsum[wv] = x;
    __syncthreads();
    int32_t before = 0;
    for (int k = 0; k < wv; ++k) before += wsum[k];
    pos[kPlanBins - 1 - j] = before + x - c;
    if (j == kPlanThreads - 1) {
      // the item count; it fits the list when the offsets meet their
      // precondition (non-decreasing, within the rows), and the list is
      // never written past its size in any case
      const int64_t cap = NH * a.n_rows;
      a.ctl[0] = static_cast<int32_t>(before + x < cap ? before + x : cap);
      for (int l = 0; l < kHeadLayers; ++l) a.ctl[1 + l] = 0;
    }
  }
  __syncthreads();
  for (int32_t r = threadIdx.x; r < a.n_req; r += kPlanThreads) {
    const int32_t nt = tiles_of(r);
    if (nt == 0) continue;
    int32_t p = atomicAdd(&pos[nt < kPlanBins ? nt : kPlanBins - 1], NH * nt);
    const int64_t cap = NH * a.n_rows;
    for (int32_t q = 0; q < nt; ++q) {
      for (int hd = 0; hd < NH; ++hd, ++p) {
        if (p >= cap) continue;
        a.items[2 * p] = r;
        a.items[2 * p + 1] = hd | (q << 2);
      }
    }
  }
}

// Output projection, residual and LayerNorm, feed-forward, residual and
// LayerNorm of a 64-row tile.
__global__ __launch_bounds__(kTileThreads) void head_ffn_kernel(HeadArgs a, int layer, const float* Hin,
                                                               float* Hout) {
  __shared__ __attribute__((aligned(16))) float sA[kTile * kSA];  // attention output, then h1
  __shared__ __attribute__((aligned(16))) float sF[kTile * kSF];  // feed-forward hidden layer
  __shared__ __attribute__((aligned(16))) float sW[FF * kSA];     // W_o, W_1, W_2 in turn (W_2 as 64 x 128)
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kTile;
  const float* Wl = a.weights + kLayer0 + layer * kLayerSize;
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  float bo[4], g1[4], be1[4], b1[FF / 16], b2[4], g2[4], be2[4];
  lane_cols(bo, Wl + kB_o);
  lane_cols(g1, Wl + kLn1g);
  lane_cols(be1, Wl + kLn1b);
  lane_cols(b1, Wl + kB_1);
  lane_cols(b2, Wl + kB_2);
  lane_cols(g2, Wl + kLn2g);
  lane_cols(be2, Wl + kLn2b);
  stage_rows(sA, a.att, r0, a.n_rows);
  stage<D, D, kSA>(sW, Wl + kW_o);
  // issued now, used after the first product: W_1 and the residual rows
  Staged<FF, D> w1;
  stage_load(w1, Wl + kW_1);
  f4 y[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = 16 * j + lane % 16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = r0 + 16 * w + 4 * (lane / 16) + r;
      y[j][r] = row < a.n_rows ? Hin[row * D + col] : 0.0f;
    }
  }
  __syncthreads();
  // y = att W_o^T + b_o + h; h1 = LN1(y)
  f4 p[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) p[j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
  tile_gemm<4, D>(sA, kSA, sW, kSA, p);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int r = 0; r < 4; ++r) y[j][r] = p[j][r] + (bo[j] + y[j][r]);
  }
  layer_norm_rows(y, g1, be1);
  __syncthreads();  // everyone is done reading sA and sW
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) sA[(16 * w + 4 * (lane / 16) + r) * kSA + 16 * j + lane % 16] = y[j][r];
  stage_store<FF, D, kSA>(sW, w1);
  __syncthreads();
  Staged<D, FF> w2;  // issued now, used after the second product
  stage_load(w2, Wl + kW_2);
  // f = relu(h1 W_1^T + b_1)
  {
    f4 f[FF / 16];
#pragma unroll
    for (int j = 0; j < FF / 16; ++j) f[j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    tile_gemm<FF / 16, D>(sA, kSA, sW, kSA, f);
#pragma unroll
    for (int j = 0; j < FF / 16; ++j) {
      const int col = 16 * j + lane % 16;
      const float bias = b1[j];
#pragma unroll
      for (int r = 0; r < 4; ++r) sF[(16 * w + 4 * (lane / 16) + r) * kSF + col] = fmaxf(f[j][r] + bias, 0.0f);
    }
  }
  __syncthreads();  // sF complete, sW free
  stage_store<D, FF, kSF>(sW, w2);
  __syncthreads();
  // z = f W_2^T + b_2 + h1; h2 = LN2(z)
  f4 z[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) z[j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
  tile_gemm<4, FF>(sF, kSF, sW, kSF, z);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int r = 0; r < 4; ++r) z[j][r] += b2[j] + y[j][r];
  }
  layer_norm_rows(z, g2, be2);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = 16 * j + lane % 16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = r0 + 16 * w + 4 * (lane / 16) + r;
      if (row < a.n_rows) Hout[row * D + col] = z[j][r];
    }
  }
}

// Mean pool of a request's rows, linear map to one logit, sigmoid. An empty
// request, or one longer than max_len, scores NaN.
constexpr int kPoolThreads = 1024;

__global__ __launch_bounds__(kPoolThreads) void head_pool_kernel(HeadArgs a, const float* H) {
  __shared__ float part[kPoolThreads / D][D];
  const int64_t req = blockIdx.x;
  const int64_t lo = a.offsets[req], hi = a.offsets[req + 1];
  const int64_t T = hi - lo;
  const int c = threadIdx.x % D, p = threadIdx.x / D;
  float s = 0.0f;
  // unrolled, so that a thread's loads are in flight together (the sum keeps
  // its order)
#pragma unroll 8
  for (int64_t r = lo + p; r < hi; r += kPoolThreads / D) s += H[r * D + c];
  part[p][c] = s;
  __syncthreads();
  if (threadIdx.x < kWave) {
    float t = 0.0f;
    for (int k = 0; k < kPoolThreads / D; ++k) t += part[k][threadIdx.x];
    const float mean = t / static_cast<float>(T > 0 ? T : 1);
    float z = mean * a.weights[kW_out + threadIdx.x];
    z = wave_sum(z) + a.weights[kB_out];
    if (threadIdx.x == 0)
      a.scores[req] = (T <= 0 || T > a.max_len) ? __uint_as_float(0x7fc00000u) : 1.0f / (1.0f + expf(-z));
  }
}

// Rows of activations, then the work list (at most kHeadHeads items per row:
// a request of T >= 1 tokens has ceil(T / 64) <= T query tiles) and the
// counters.
size_t head_workspace_bytes(int64_t n_rows) {
  return static_cast<size_t>(n_rows) * ((2 * D + QKV + D) * sizeof(float) + 2 * NH * sizeof(int32_t)) +
         static_cast<size_t>(1 + kHeadLayers) * sizeof(int32_t);
}

hipError_t launch_head(const HeadArgs& args, hipStream_t stream) {
  if (args.n_req == 0) return hipSuccess;
  HeadArgs a = args;
  float* H0 = a.ws;
  float* H1 = H0 + a.n_rows * D;
  a.qkv = H1 + a.n_rows * D;
  a.att = a.qkv + a.n_rows * QKV;
  a.items = reinterpret_cast<int32_t*>(a.att + a.n_rows * D);
  a.ctl = a.items + 2 * NH * a.n_rows;
  const unsigned tiles = static_cast<unsigned>((a.n_rows + kTile - 1) / kTile);
  // persistent attention workgroups: two per CU of this part, fewer when
  // there are fewer items than that
  const int64_t max_items = NH * a.n_rows;
  const unsigned attn_grid = static_cast<unsigned>(max_items < kAttnPersist ? max_items : kAttnPersist);
  if (a.n_rows > 0) {
    head_plan_kernel<<<1, kPlanThreads, 0, stream>>>(a);
    float* Hin = H0;
    float* Hout = H1;
    for (int l = 0; l < kHeadLayers; ++l) {
      if (l == 0)
        head_qkv_kernel<true><<<tiles, kTileThreads, 0, stream>>>(a, 0, nullptr, Hin);
      else
        head_qkv_kernel<false><<<tiles, kTileThreads, 0, stream>>>(a, l, Hin, nullptr);
      head_attn_kernel<<<attn_grid, kAttnWaves * kWave, 0, stream>>>(a, l);
      head_ffn_kernel<<<tiles, kTileThreads, 0, stream>>>(a, l, Hin, Hout);
      float* t = Hin;
      Hin = Hout;
      Hout = t;
    }
    head_pool_kernel<<<static_cast<unsigned>(a.n_req), kPoolThreads, 0, stream>>>(a, Hin);
  } else {
    head_pool_kernel<<<static_cast<unsigned>(a.n_req), kPoolThreads, 0, stream>>>(a, H0);
  }
  return hipGetLastError();
}

}  // namespace pr
