// kernels.hpp -- launch interface between the host ABI (api.cpp) and the
// HIP kernels.  Plain structs of device pointers and sizes; the host side
// has already validated every size and pointer it can see.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace sla {

struct PendingArgs {
  const void *k;          // [B][np][H][dk] activation dtype
  const float *u;         // [B][np][H][dv]
  const float *alpha;     // [B][np][H] ([B][np][H][dk]: per-key gates)
  const int32_t *parent;  // [B][np]
  int32_t n;              // np
  const int32_t *path;    // [B][np]
  const int32_t *len;     // [B]
};

struct VerifyArgs {
  int32_t B, H, dk, dv, n;
  int32_t family;   // SLA_FAMILY_*: which of alpha, beta the step reads, and the gate layout
  bool chain;
  bool has_pending;
  bool late_state;  // parallel route: issue the state reads after the first barrier
  bool stagger;     // parallel route: hold the state reads back briefly (a full round of workgroups)
  bool write_through;  // 1-node kernel: committed rows written through at device scope
  bool xcd_group;      // 1-node kernel: a unit's slabs numbered back to back on one XCD
  float *state;
  PendingArgs pend;
  const void *q, *k, *v;
  const float *alpha, *beta;
  const int32_t *parent;
  float *out;
  void *fk;
  float *fu;
  float *falpha;
  int32_t *fparent;
  int32_t *status;
};

struct CommitArgs {
  int32_t B, H, dk, dv, n;
  bool gate_vec;       // alpha holds dk gates per record (GLA) instead of one
  bool write_through;  // state rows written through at device scope (at least one workgroup per CU)
  bool xcd_group;      // a unit's slabs numbered back to back on one XCD
  float *state;
  const void *k;
  const float *u;
  const float *alpha;
  const int32_t *parent;
  const int32_t *path;
  const int32_t *len;
  int32_t *status;
};

struct TopologyArgs {
  int32_t B, n;
  const int32_t *parent;
  int32_t *depth;
  uint64_t *anc;
  int32_t *order;
  int32_t *n_children;
  int32_t *status;
};

// Each launcher returns hipSuccess or the launch error.  `dtype` is
// SLA_DTYPE_F32 or SLA_DTYPE_BF16.
hipError_t launch_verify_serial(const VerifyArgs &a, int dtype, hipStream_t s);
// chain-decomposed hybrid (chains run through the serial kernel)
hipError_t launch_verify_hybrid(const VerifyArgs &a, int dtype, hipStream_t s);
bool parallel_supported(int dk, int dv, int n, int dtype);
hipError_t launch_verify_parallel(const VerifyArgs &a, int dtype, hipStream_t s);
// 1-node drafts (a.n == 1), any family and activation dtype
hipError_t launch_verify_decode(const VerifyArgs &a, int dtype, hipStream_t s);
hipError_t launch_commit(const CommitArgs &a, int dtype, hipStream_t s);
hipError_t launch_topology(const TopologyArgs &a, hipStream_t s);

}  // namespace sla
