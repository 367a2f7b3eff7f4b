// treewy_path_from_node kernel: root-to-node path of each sequence's accepted
// node (the accepted node's ancestors and itself, Method eq. 3), one thread
// per sequence.  Integer work only, so the result is exact.
#include "device.h"
#include "launch.h"

namespace treewy {

__global__ __launch_bounds__(THREADS) void path_from_node_kernel(
    const int32_t *__restrict__ parent, const int32_t *__restrict__ accepted, int N, int B,
    int L_max, int32_t *__restrict__ path, int32_t *__restrict__ path_len,
    int32_t *__restrict__ err) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int32_t *par = parent + (size_t)b * N;
    int32_t *out = path + (size_t)b * L_max;
    const int a = accepted[b];
    int len = 0;
    bool ok = a >= -1 && a < N;
    // Count the path length first; each step must move to a smaller index.
    for (int cur = ok ? a : -1; cur >= 0;) {
        const int p = par[cur];
        if (p < -1 || p >= cur || ++len > L_max) {
            ok = false;
            break;
        }
        cur = p;
    }
    if (!ok) {
        len = 0;
        flag_error(err, b, TREEWY_FLAG_BAD_PATH);
    }
    int cur = a;
    for (int l = len - 1; l >= 0; --l) {
        out[l] = cur;
        cur = par[cur];
    }
    for (int l = len; l < L_max; ++l) out[l] = -1;
    path_len[b] = len;
}

hipError_t launch_path_from_node(const int32_t *parent, const int32_t *accepted, int N, int B,
                                 int L_max, int32_t *path, int32_t *path_len, int32_t *err,
                                 hipStream_t stream) {
    const int blocks = (B + THREADS - 1) / THREADS;
    hipLaunchKernelGGL(path_from_node_kernel, dim3((unsigned)blocks), dim3(THREADS), 0, stream,
                       parent, accepted, N, B, L_max, path, path_len, err);
    return hipGetLastError();
}

}  // namespace treewy
