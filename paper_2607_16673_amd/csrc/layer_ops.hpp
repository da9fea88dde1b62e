// layer_ops.hpp -- launch interface between the host ABI (api.cpp) and the
// kernels around the recurrent core: the short causal convolution with its
// conv state, and draft pruning / packing.  Plain structs of device pointers
// and sizes; the host side has already validated what it can see.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace sla {

// Short causal convolution.  For the verify kernel, path/len/pend_* describe
// the pending commit (has_pending); for the commit kernel, x and parent are
// the draft the accepted path came from and path/len the path itself.
struct ConvArgs {
  int32_t B, D, K, n;
  int32_t activation;
  bool has_pending;
  float *conv_state;      // [B][K-1][D]
  const void *x;          // [B][n][D] activation dtype
  const float *weight;    // [D][K]
  const float *bias;      // [D] or null
  const int32_t *parent;  // [B][n]
  void *y;                // [B][n][D] activation dtype
  const void *pend_x;     // [B][pend_n][D]
  const int32_t *pend_parent;  // [B][pend_n]
  int32_t pend_n;
  const int32_t *path;    // [B][pend_n] (verify) or [B][n] (commit)
  const int32_t *len;     // [B]
  int32_t *status;
};

// Draft pruning and packing, one sequence per wavefront (n <= 64).
struct PruneArgs {
  int32_t B, n;
  float tau;
  int32_t budget;            // <= 0: no budget
  const int32_t *parent;     // [B][n]
  const float *logp;         // [B][n]
  int32_t *packed_parent;    // [B][n]
  int32_t *index_map;        // [B][n]
  int32_t *count;            // [B]
  float *scores;             // [B][n] or null
  int32_t *status;           // [B] or null
};

struct MaskArgs {
  int32_t B, n;
  const uint64_t *mask;  // [B][n] rows
  int32_t *parent;       // [B][n]
  int32_t *status;       // [B] or null
};

hipError_t launch_conv(const ConvArgs &a, int dtype, bool commit, hipStream_t s);
hipError_t launch_prune(const PruneArgs &a, hipStream_t s);
hipError_t launch_mask_to_parent(const MaskArgs &a, hipStream_t s);

}  // namespace sla
