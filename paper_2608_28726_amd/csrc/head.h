// Launch interface of the verifier-head kernels (internal).
#pragma once

#include "device_util.h"

namespace pr {

constexpr int kHeadD = 64;        // model width
constexpr int kHeadFF = 128;      // feed-forward width
constexpr int kHeadHeads = 4;     // attention heads (16 dimensions each)
constexpr int kHeadLayers = 2;    // encoder layers
constexpr int kHeadWeights = 67329;

struct HeadArgs {
  const float* X;          // [n_rows][4] input sequence (l, m, h, rho)
  int64_t n_rows;
  const int32_t* offsets;  // [n_req + 1]
  int32_t n_req;
  int32_t max_len;         // longest request the attention grid covers
  const float* weights;    // [kHeadWeights]
  float* scores;           // [n_req]
  float* ws;               // workspace: H0, H1 [n_rows][64], qkv [n_rows][192], att [n_rows][64],
                           // then the attention work list and its counters
  float* qkv;              // set by launch_head
  float* att;              // set by launch_head
  int32_t* items;          // set by launch_head: [2][n_rows * kHeadHeads] work items (request; head | tile << 2)
  int32_t* ctl;            // set by launch_head: [0] item count, [1 + l] next item of layer l
};

size_t head_workspace_bytes(int64_t n_rows);
hipError_t launch_head(const HeadArgs& a, hipStream_t stream);

}  // namespace pr
