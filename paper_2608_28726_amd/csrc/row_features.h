// Launch interface of the row-reduction and top-p kernels (internal).
#pragma once

#include "device_util.h"

namespace pr {

// Device-resident state of the streaming decode variant, one entry per slot.
struct StreamDev {
  int32_t max_slots;
  int32_t max_len;
  int32_t* count;     // [max_slots] tokens seen
  uint32_t* nanbits;  // [max_slots] bit f set: a NaN value of feature f was seen
  double* sum;        // [max_slots][4] running sums of A
  float* minv;        // [max_slots][4] running minima of A (+inf when empty)
  float* hist;        // [max_slots][4][max_len] every token's A, for the exact quantile
  // Bounded-memory mode (max_len == 0, hist NULL): P-square markers instead
  // of the history.
  double* p2q;        // [max_slots][5][4] marker heights, NULL otherwise
  int32_t* p2n;       // [max_slots][4][4] positions of markers 1..3, observations fed
  double p2p;         // the quantile they track
};

// What the merge of a split row needs from the row besides the partial
// states: written by the row's first workgroup.
struct RowMeta {
  float T;       // temperature
  float zy;      // logit of the sampled token (NaN when the id is invalid)
  int32_t y;     // sampled id, -1 when invalid
  uint32_t fix;  // rank corrections the vector loop leaves out
};

struct RowArgs {
  const void* logits;
  int64_t n_rows;
  int32_t V;
  int64_t row_stride;
  const int32_t* sampled_ids;
  const float* temperature;
  const float* top_p;
  pr_token_features_t out;  // max_logit == NULL: outputs not written (streaming only)
  int G;                    // workgroups per row
  Partial* ws;              // [n_rows][G] partial states when G > 1, then RowMeta [n_rows]
  const int32_t* slot_ids;  // streaming only (NULL offline)
  StreamDev st;             // streaming only
  // The paper's verifier input sequence (NULL X: not computed).
  float* X;                 // [n_rows][4]: (l, m, h, rho)
  const int32_t* offsets;   // [n_req + 1] request boundaries
  int32_t n_req;
  int32_t top_k;            // K of the top-K entropy, 1..topk::kMaxK
  // Fused sampling (sampled_ids NULL): the drawn token of each row.
  int32_t* sampled_out;     // [n_rows]
  uint32_t key0, key1;      // generator key from the caller's seed and offset
};

// Workgroups per row chosen for a shape (the same in every call, so that the
// workspace size query and the launch agree).
int row_split(int64_t n_rows, int32_t V, pr_dtype dtype);

// Bytes of split-row workspace for n_rows rows of G workgroups each.
inline size_t split_workspace_bytes(int64_t n_rows, int G) {
  return G > 1 ? static_cast<size_t>(n_rows) * (static_cast<size_t>(G) * sizeof(Partial) + sizeof(RowMeta)) : 0;
}

// The RowMeta records after the partial states.
__host__ __device__ inline RowMeta* split_meta(Partial* ws, int64_t n_rows, int G) {
  return reinterpret_cast<RowMeta*>(ws + n_rows * G);
}

// One kernel when G == 1, partial-state and merge kernels otherwise; with
// slot ids (streaming) each finalised row also updates its request slot.
hipError_t launch_row_features(const RowArgs& a, pr_dtype dtype, hipStream_t stream);

// The verifier input sequence X (with the features when a.out is set): one
// workgroup per row, no split.
hipError_t launch_feature_sequence(const RowArgs& a, pr_dtype dtype, hipStream_t stream);

// Fused sample-and-verify: each row's token is drawn in the same pass
// (a.sampled_out), then its features (a.out, when set) and row of X (a.X,
// when set) are written as for that token. One workgroup per row.
hipError_t launch_sample(const RowArgs& a, pr_dtype dtype, hipStream_t stream);

}  // namespace pr
