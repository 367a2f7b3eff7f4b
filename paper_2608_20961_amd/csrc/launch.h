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

// One chunk of the chain prefill: commit the previous chunk (n_prev tokens,
// n_prev < 0 for none) into the state, then verify this chunk (n tokens) as
// a chain.  Inputs are slices of [B, H, T, ...] tensors; U is [B, H, 64, d_v].
hipError_t launch_prefill_chunk(const void *S_old, const float *U_prev, const void *k_prev,
                                const float *alpha_prev, int n_prev, const void *q, const void *k,
                                const void *v, const float *alpha, const float *beta, int n, int T, int B,
                                int H, bool f32_in, bool bf16_state, void *S_new, void *o, float *U,
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
