// C ABI of libtreewy.so: host-side argument checks, then one kernel launch on
// the caller's stream.  Declared in include/treewy.h.
#include <stdint.h>

#include "device.h"
#include "launch.h"

namespace {

constexpr int kMaxTree = treewy::MAX_TREE;   // verify, commit and the tree helpers
constexpr int kMaxOnePass = 64;              // the fused call and the snapshot baseline

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

treewy_status hip_status(hipError_t e) { return e == hipSuccess ? TREEWY_OK : TREEWY_ERR_HIP; }

// Shared checks for the calls that take the full verify inputs.
// The state is fp32, or bf16 with bf16 inputs.
treewy_status check_state(treewy_dtype state, treewy_dtype in) {
    if (state != TREEWY_F32 && state != TREEWY_BF16) return TREEWY_ERR_INVALID_ARG;
    if (state == TREEWY_BF16 && in != TREEWY_BF16) return TREEWY_ERR_UNSUPPORTED;
    return TREEWY_OK;
}

treewy_status check_common(int N, int B, int H, int d_k, int d_v, treewy_dtype dt, int max_n) {
    if (B < 0 || H < 0 || N < 0) return TREEWY_ERR_INVALID_ARG;
    if (dt != TREEWY_F32 && dt != TREEWY_BF16) return TREEWY_ERR_INVALID_ARG;
    if (d_k != treewy::D || d_v != treewy::D) return TREEWY_ERR_UNSUPPORTED;
    if (N > max_n) return TREEWY_ERR_UNSUPPORTED;
    if ((int64_t)B * H > INT32_MAX) return TREEWY_ERR_UNSUPPORTED;
    return TREEWY_OK;
}

}  // namespace

extern "C" {

treewy_status treewy_verify(const void *S0, const void *q, const void *k, const void *v,
                            const float *alpha, const float *beta, const int32_t *parent, int N,
                            int B, int H, int d_k, int d_v, treewy_dtype in_dtype, treewy_dtype state_dtype,
                            void *o, float *U, int32_t *err, void *stream) {
    treewy_status st = check_common(N, B, H, d_k, d_v, in_dtype, kMaxTree);
    if (st == TREEWY_OK) st = check_state(state_dtype, in_dtype);
    if (st != TREEWY_OK) return st;
    if (N == 0 || B == 0 || H == 0) return TREEWY_OK;
    if (!S0 || !q || !k || !v || !alpha || !beta || !parent || !o || !U) return TREEWY_ERR_INVALID_ARG;
    if (!aligned16(S0) || !aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) ||
        !aligned16(U))
        return TREEWY_ERR_INVALID_ARG;
    return hip_status(treewy::launch_verify(S0, q, k, v, alpha, beta, parent, N, B, H,
                                            in_dtype == TREEWY_F32, state_dtype == TREEWY_BF16, o, U, err,
                                            static_cast<hipStream_t>(stream)));
}

treewy_status treewy_commit(const void *S0, const float *U, const void *k, const float *alpha,
                            const int32_t *path, const int32_t *path_len, int L_max,
                            const int32_t *parent, int N, int B, int H, int d_k, int d_v,
                            treewy_dtype k_dtype, treewy_dtype state_dtype, void *S_new, int32_t *err,
                            void *stream) {
    treewy_status st = check_common(N, B, H, d_k, d_v, k_dtype, kMaxTree);
    if (st == TREEWY_OK && state_dtype != TREEWY_F32 && state_dtype != TREEWY_BF16) st = TREEWY_ERR_INVALID_ARG;
    if (st != TREEWY_OK) return st;
    if (L_max < 0) return TREEWY_ERR_INVALID_ARG;
    if (L_max > kMaxTree) return TREEWY_ERR_UNSUPPORTED;
    if (B == 0 || H == 0) return TREEWY_OK;
    if (!S0 || !path_len || !S_new) return TREEWY_ERR_INVALID_ARG;
    if (N > 0 && (!U || !k || !alpha)) return TREEWY_ERR_INVALID_ARG;
    if (L_max > 0 && !path) return TREEWY_ERR_INVALID_ARG;
    if (!aligned16(S0) || !aligned16(S_new)) return TREEWY_ERR_INVALID_ARG;
    return hip_status(treewy::launch_commit(S0, U, k, alpha, path, path_len, L_max, parent, N, B, H,
                                            k_dtype == TREEWY_F32, state_dtype == TREEWY_BF16, S_new, err,
                                            static_cast<hipStream_t>(stream)));
}

treewy_status treewy_commit_verify(const void *S_old, const float *U_prev, const void *k_prev,
                                   const float *alpha_prev, const int32_t *path,
                                   const int32_t *path_len, int L_max, const int32_t *parent_prev,
                                   int N_prev, const void *q, const void *k, const void *v,
                                   const float *alpha, const float *beta, const int32_t *parent,
                                   int N, int B, int H, int d_k, int d_v, treewy_dtype in_dtype,
                                   treewy_dtype state_dtype, void *S_new, void *o, float *U, int32_t *err,
                                   void *stream) {
    treewy_status st = check_common(N, B, H, d_k, d_v, in_dtype, kMaxOnePass);
    if (st == TREEWY_OK) st = check_state(state_dtype, in_dtype);
    if (st != TREEWY_OK) return st;
    if (N_prev < 0 || L_max < 0) return TREEWY_ERR_INVALID_ARG;
    if (N_prev > kMaxOnePass || L_max > kMaxOnePass) return TREEWY_ERR_UNSUPPORTED;
    if (B == 0 || H == 0) return TREEWY_OK;
    if (!S_old || !path_len || !S_new) return TREEWY_ERR_INVALID_ARG;
    if (N_prev > 0 && (!U_prev || !k_prev || !alpha_prev)) return TREEWY_ERR_INVALID_ARG;
    if (L_max > 0 && !path) return TREEWY_ERR_INVALID_ARG;
    if (N > 0 && (!q || !k || !v || !alpha || !beta || !parent || !o || !U)) return TREEWY_ERR_INVALID_ARG;
    if (!aligned16(S_old) || !aligned16(S_new) || !aligned16(U_prev) || !aligned16(k_prev) ||
        !aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(U))
        return TREEWY_ERR_INVALID_ARG;
    // U over U_prev is safe only row block for row block (each unit reads its
    // previous rows before it writes its new ones).
    if (N > 0 && U == U_prev && N != N_prev) return TREEWY_ERR_INVALID_ARG;
    return hip_status(treewy::launch_commit_verify(S_old, U_prev, k_prev, alpha_prev, path, path_len, L_max,
                                                   parent_prev, N_prev, q, k, v, alpha, beta, parent, N, B,
                                                   H, in_dtype == TREEWY_F32, state_dtype == TREEWY_BF16, S_new,
                                                   o, U, err, static_cast<hipStream_t>(stream)));
}

treewy_status treewy_chain_prefill(const void *S0, const void *q, const void *k, const void *v,
                                   const float *alpha, const float *beta, int T, int B, int H, int d_k, int d_v,
                                   treewy_dtype in_dtype, treewy_dtype state_dtype, void *S_T, void *o,
                                   int32_t *err, void *stream) {
    if (T < 0) return TREEWY_ERR_INVALID_ARG;
    treewy_status st = check_common(0, B, H, d_k, d_v, in_dtype, kMaxTree);
    if (st == TREEWY_OK) st = check_state(state_dtype, in_dtype);
    if (st != TREEWY_OK) return st;
    if ((int64_t)T * B * H > INT32_MAX) return TREEWY_ERR_UNSUPPORTED;
    if (B == 0 || H == 0) return TREEWY_OK;
    if (!S0 || !S_T) return TREEWY_ERR_INVALID_ARG;
    if (T > 0 && (!q || !k || !v || !alpha || !beta || !o)) return TREEWY_ERR_INVALID_ARG;
    if (!aligned16(S0) || !aligned16(S_T) || !aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
        return TREEWY_ERR_INVALID_ARG;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (T == 0) {
        const size_t bytes = (size_t)B * H * treewy::D * treewy::D * (state_dtype == TREEWY_BF16 ? 2 : 4);
        return S_T == S0 ? TREEWY_OK : hip_status(hipMemcpyAsync(S_T, S0, bytes, hipMemcpyDeviceToDevice, s));
    }
    return hip_status(treewy::launch_prefill(S0, q, k, v, alpha, beta, T, B, H, in_dtype == TREEWY_F32,
                                             state_dtype == TREEWY_BF16, S_T, o, err, s));
}

treewy_status treewy_snapshot_verify(const float *S0, const void *q, const void *k, const void *v,
                                     const float *alpha, const float *beta, const int32_t *parent,
                                     int N, int B, int H, int d_k, int d_v, treewy_dtype in_dtype,
                                     void *o, float *snapshots, int32_t *err, void *stream) {
    treewy_status st = check_common(N, B, H, d_k, d_v, in_dtype, kMaxOnePass);
    if (st != TREEWY_OK) return st;
    if (N == 0 || B == 0 || H == 0) return TREEWY_OK;
    if (!S0 || !q || !k || !v || !alpha || !beta || !parent || !o || !snapshots)
        return TREEWY_ERR_INVALID_ARG;
    if (!aligned16(S0) || !aligned16(snapshots)) return TREEWY_ERR_INVALID_ARG;
    return hip_status(treewy::launch_snapshot_verify(S0, q, k, v, alpha, beta, parent, N, B, H,
                                                     in_dtype == TREEWY_F32, o, snapshots, err,
                                                     static_cast<hipStream_t>(stream)));
}

treewy_status treewy_snapshot_commit(const float *S0, const float *snapshots, const int32_t *accepted,
                                     int N, int B, int H, int d_k, int d_v, float *S_new,
                                     int32_t *err, void *stream) {
    treewy_status st = check_common(N, B, H, d_k, d_v, TREEWY_F32, kMaxOnePass);
    if (st != TREEWY_OK) return st;
    if (B == 0 || H == 0) return TREEWY_OK;
    if (!S0 || !accepted || !S_new || (N > 0 && !snapshots)) return TREEWY_ERR_INVALID_ARG;
    if (!aligned16(S0) || !aligned16(S_new) || (snapshots && !aligned16(snapshots)))
        return TREEWY_ERR_INVALID_ARG;
    return hip_status(treewy::launch_snapshot_commit(S0, snapshots, accepted, N, B, H, S_new, err,
                                                     static_cast<hipStream_t>(stream)));
}

treewy_status treewy_path_from_node(const int32_t *parent, const int32_t *accepted, int N, int B,
                                    int L_max, int32_t *path, int32_t *path_len, int32_t *err,
                                    void *stream) {
    if (N < 0 || B < 0 || L_max < 0) return TREEWY_ERR_INVALID_ARG;
    if (N > kMaxTree || L_max > kMaxTree) return TREEWY_ERR_UNSUPPORTED;
    if (B == 0) return TREEWY_OK;
    if (!accepted || !path_len || (N > 0 && !parent) || (L_max > 0 && !path))
        return TREEWY_ERR_INVALID_ARG;
    return hip_status(treewy::launch_path_from_node(parent, accepted, N, B, L_max, path, path_len,
                                                    err, static_cast<hipStream_t>(stream)));
}

treewy_status treewy_accept_greedy(const int32_t *parent, const int32_t *draft_token,
                                   const int32_t *target_token, const int32_t *root_token, int N, int B,
                                   int L_max, int32_t *path, int32_t *path_len, int32_t *bonus,
                                   int32_t *err, void *stream) {
    if (N < 0 || B < 0 || L_max < 0) return TREEWY_ERR_INVALID_ARG;
    if (N > kMaxTree || L_max > kMaxTree) return TREEWY_ERR_UNSUPPORTED;
    if (B == 0) return TREEWY_OK;
    if (!root_token || !path_len || (N > 0 && (!parent || !draft_token || !target_token)) ||
        (L_max > 0 && !path))
        return TREEWY_ERR_INVALID_ARG;
    return hip_status(treewy::launch_accept_greedy(parent, draft_token, target_token, root_token, N, B, L_max,
                                                   path, path_len, bonus, err,
                                                   static_cast<hipStream_t>(stream)));
}

const char *treewy_status_string(treewy_status status) {
    switch (status) {
    case TREEWY_OK: return "ok";
    case TREEWY_ERR_INVALID_ARG: return "invalid argument (null or misaligned pointer, bad size or dtype)";
    case TREEWY_ERR_UNSUPPORTED:
        return "unsupported size or dtype (d_k, d_v must be 128; N, L_max at most 256, and 64 for the fused call "
               "and the snapshot baseline; a bf16 state needs bf16 inputs)";
    case TREEWY_ERR_HIP: return "HIP launch failed";
    }
    return "unknown status";
}

}  // extern "C"
