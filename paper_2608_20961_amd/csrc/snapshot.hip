// Full-state-snapshotting baseline (the paper's approach (i), "storeall"):
// run the gated delta rule (eq. 1) node by node and write every node's full
// state, so that rollback is a copy of one snapshot.  Kept deliberately as the
// store-all data flow, for the memory and bandwidth comparison with
// reconstruct-on-commit; it is not the method.
//
// One workgroup per (sequence, head) keeps the running 128 x 128 fp32 state in
// registers: thread t holds rows t/32 + 8i (i < 16) at columns 4(t%32)..+3, so
// every state load and store instruction of the workgroup covers 4 KiB of
// contiguous HBM.  A node whose parent is not the previous node reloads the
// parent's snapshot (its own elements, written earlier by the same thread).
#include "device.h"
#include "launch.h"

namespace treewy {

template <bool F32IN>
__global__ __launch_bounds__(THREADS) void snapshot_verify_kernel(
    const float *__restrict__ S0, const void *__restrict__ q_, const void *__restrict__ k_,
    const void *__restrict__ v_, const float *__restrict__ alpha, const float *__restrict__ beta,
    const int32_t *__restrict__ parent, int N, int H, void *__restrict__ o_,
    float *__restrict__ snaps, int32_t *__restrict__ err) {
    using In = typename std::conditional<F32IN, float, __bf16>::type;
    __shared__ __attribute__((aligned(16))) float k_s[D];
    __shared__ __attribute__((aligned(16))) float q_s[D];
    __shared__ float v_s[D];
    __shared__ int p_s;
    const In *q = static_cast<const In *>(q_);
    const In *k = static_cast<const In *>(k_);
    const In *v = static_cast<const In *>(v_);
    In *o = static_cast<In *>(o_);

    const int tid = threadIdx.x, u = blockIdx.x, b = u / H;
    const int r0 = tid >> 5, c4 = (tid & 31) * 4, lane32 = tid & 31;
    const size_t node0 = (size_t)u * N;
    const f32x4 *s0 = reinterpret_cast<const f32x4 *>(S0 + (size_t)u * D * D);
    f32x4 s[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) s[i] = s0[tid + THREADS * i];

    for (int t = 0; t < N; ++t) {
        __syncthreads();                                  // previous node done with k_s/q_s/v_s
        if (tid < D) {
            const size_t row = (node0 + t) * D + tid;
            k_s[tid] = to_f32(k[row]);
            q_s[tid] = to_f32(q[row]);
            v_s[tid] = to_f32(v[row]);
        }
        if (tid == 0) {
            int p = parent[(size_t)b * N + t];
            if (p < -1 || p >= t) {
                flag_error(err, b, TREEWY_FLAG_BAD_PARENT);
                p = -1;
            }
            p_s = p;
        }
        __syncthreads();
        const int p = p_s;
        if (p != t - 1) {
            const f32x4 *from = p < 0 ? s0 : reinterpret_cast<const f32x4 *>(snaps + (node0 + p) * D * D);
            __threadfence_block();                        // this thread's earlier snapshot stores first
#pragma unroll
            for (int i = 0; i < 16; ++i) s[i] = from[tid + THREADS * i];
        }
        const f32x4 kk = *reinterpret_cast<const f32x4 *>(k_s + c4);
        const f32x4 qq = *reinterpret_cast<const f32x4 *>(q_s + c4);
        float sk[16], sq[16];
        float kq = kk[0] * qq[0] + kk[1] * qq[1] + kk[2] * qq[2] + kk[3] * qq[3];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            sk[i] = s[i][0] * kk[0] + s[i][1] * kk[1] + s[i][2] * kk[2] + s[i][3] * kk[3];
            sq[i] = s[i][0] * qq[0] + s[i][1] * qq[1] + s[i][2] * qq[2] + s[i][3] * qq[3];
        }
        // Sum over the 32 lanes that share these rows.
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) {
            kq += __shfl_xor(kq, off, 32);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                sk[i] += __shfl_xor(sk[i], off, 32);
                sq[i] += __shfl_xor(sq[i], off, 32);
            }
        }
        const float al = alpha[node0 + t], be = beta[node0 + t];
        f32x4 *snap = reinterpret_cast<f32x4 *>(snaps + (node0 + t) * D * D);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int r = r0 + 8 * i;
            const float vt = be * (v_s[r] - al * sk[i]);           // pseudo-value of row r
            s[i] = al * s[i] + vt * kk;                            // eq. 1 via the key rewrite
            if (lane32 == 0) o[(node0 + t) * D + r] = from_f32<In>(al * sq[i] + vt * kq);
            snap[tid + THREADS * i] = s[i];
        }
    }
}

__global__ __launch_bounds__(THREADS) void snapshot_commit_kernel(
    const float *S0, const float *__restrict__ snaps, const int32_t *__restrict__ accepted, int N,
    int H, float *S_new, int32_t *__restrict__ err) {
    const int tid = threadIdx.x, u = blockIdx.x, b = u / H;
    int a = accepted[b];
    if (a < -1 || a >= N) {
        if (tid == 0 && u % H == 0) flag_error(err, b, TREEWY_FLAG_BAD_PATH);
        a = -1;
    }
    const f32x4 *from = reinterpret_cast<const f32x4 *>(
        a < 0 ? S0 + (size_t)u * D * D : snaps + ((size_t)u * N + a) * D * D);
    f32x4 *dst = reinterpret_cast<f32x4 *>(S_new + (size_t)u * D * D);
    f32x4 s[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) s[i] = from[tid + THREADS * i];
#pragma unroll
    for (int i = 0; i < 16; ++i) dst[tid + THREADS * i] = s[i];
}

hipError_t launch_snapshot_verify(const float *S0, const void *q, const void *k, const void *v,
                                  const float *alpha, const float *beta, const int32_t *parent,
                                  int N, int B, int H, bool f32_in, void *o, float *snapshots,
                                  int32_t *err, hipStream_t stream) {
    const dim3 grid((unsigned)(B * H)), block(THREADS);
    if (f32_in)
        hipLaunchKernelGGL((snapshot_verify_kernel<true>), grid, block, 0, stream, S0, q, k, v, alpha,
                           beta, parent, N, H, o, snapshots, err);
    else
        hipLaunchKernelGGL((snapshot_verify_kernel<false>), grid, block, 0, stream, S0, q, k, v, alpha,
                           beta, parent, N, H, o, snapshots, err);
    return hipGetLastError();
}

hipError_t launch_snapshot_commit(const float *S0, const float *snapshots, const int32_t *accepted,
                                  int N, int B, int H, float *S_new, int32_t *err,
                                  hipStream_t stream) {
    hipLaunchKernelGGL(snapshot_commit_kernel, dim3((unsigned)(B * H)), dim3(THREADS), 0, stream, S0,
                       snapshots, accepted, N, H, S_new, err);
    return hipGetLastError();
}

}  // namespace treewy
