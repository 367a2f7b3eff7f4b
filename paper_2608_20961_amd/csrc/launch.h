// Kernel launchers behind the C ABI.  Arguments are already validated by the
// caller; each returns the HIP error of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace treewy {

hipError_t launch_verify(const void *S0, const void *q, const void *k, const void *v,
                         const float *alpha, const float *beta, const int32_t *parent, int N,
                         int B, int H, bool f32_in, bool bf16_state, void *o, float *U, int32_t *err,
                         hipStream_t stream);

// Commit of the previous round's accepted path fused into this round's verify.
hipError_t launch_commit_verify(const void *S_old, const float *U_prev, const void *k_prev,
                                const float *alpha_prev, const int32_t *path, const int32_t *path_len,
                                int L_max, const int32_t *parent_prev, int N_prev, const void *q,
                                const void *k, const void *v, const float *alpha, const float *beta,
                                const int32_t *parent, int N, int B, int H, bool f32_in, bool bf16_state,
                                void *S_new, void *o, float *U, int32_t *err, hipStream_t stream);

// Chain prefill: T tokens per unit in chunks of 64, one launch, the state in
// registers between chunks; inputs and o are [B, H, T, ...].
hipError_t launch_prefill(const void *S0, const void *q, const void *k, const void *v, const float *alpha,
                          const float *beta, int T, int B, int H, bool f32_in, bool bf16_state, void *S_T, void *o,
                          int32_t *err, hipStream_t stream);

hipError_t launch_commit(const void *S0, const float *U, const void *k, const float *alpha,
                         const int32_t *path, const int32_t *path_len, int L_max,
                         const int32_t *parent, int N, int B, int H, bool f32_k, bool bf16_state,
                         void *S_new, int32_t *err, hipStream_t stream);

hipError_t launch_snapshot_verify(const float *S0, const void *q, const void *k, const void *v,
                                  const float *alpha, const float *beta, const int32_t *parent,
                                  int N, int B, int H, bool f32_in, void *o, float *snapshots,
                                  int32_t *err, hipStream_t stream);

hipError_t launch_snapshot_commit(const float *S0, const float *snapshots, const int32_t *accepted,
                                  int N, int B, int H, float *S_new, int32_t *err,
                                  hipStream_t stream);

hipError_t launch_path_from_node(const int32_t *parent, const int32_t *accepted, int N, int B,
                                 int L_max, int32_t *path, int32_t *path_len, int32_t *err,
                                 hipStream_t stream);

hipError_t launch_accept_greedy(const int32_t *parent, const int32_t *draft, const int32_t *target,
                                const int32_t *root, int N, int B, int L_max, int32_t *path,
                                int32_t *path_len, int32_t *bonus, int32_t *err, hipStream_t stream);

}  // namespace treewy
