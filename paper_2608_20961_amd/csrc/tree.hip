// Tree helpers, integer work only (results are exact):
//  - treewy_path_from_node: root-to-node path of each sequence's accepted node
//    (the accepted node's ancestors and itself, Method eq. 3), one thread per
//    sequence;
//  - treewy_accept_greedy: greedy acceptance of the draft tree, one wave per
//    sequence with lane t holding nodes t, t + 64, t + 128 and t + 192.
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

// Greedy acceptance (Background: the target keeps the longest run of draft
// tokens it would have generated itself; the paper verifies greedily,
// Implementation).  From the committed prefix, repeatedly move to the child
// whose draft token equals the target's prediction at the current position
// (lowest index among equal siblings) until no child matches.  Children have
// larger indices than their parent, so the walk ends within N steps.
template <int W>                                        // nodes per lane: lane + 64 w, w < W
__global__ __launch_bounds__(THREADS) void accept_greedy_kernel(
    const int32_t *__restrict__ parent, const int32_t *__restrict__ draft,
    const int32_t *__restrict__ target, const int32_t *__restrict__ root, int N, int B, int L_max,
    int32_t *__restrict__ path, int32_t *__restrict__ path_len, int32_t *__restrict__ bonus,
    int32_t *__restrict__ err) {
    const int lane = threadIdx.x & 63;
    const int b = blockIdx.x * (THREADS / 64) + (threadIdx.x >> 6);
    if (b >= B) return;                                  // whole waves leave together
    const size_t row = (size_t)b * N;
    int par[W], tok[W], pred[W];
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int t = lane + 64 * w;
        par[w] = -1;
        tok[w] = pred[w] = 0;
        if (t < N) {
            par[w] = parent[row + t];
            tok[w] = draft[row + t];
            pred[w] = target[row + t];
            if (par[w] < -1 || par[w] >= t) {
                flag_error(err, b, TREEWY_FLAG_BAD_PARENT);
                par[w] = -1;
            }
        }
    }
    int pos = -1, want = root[b], len = 0;
    int mine[W];                                         // entry lane + 64 w of the accepted path
#pragma unroll
    for (int w = 0; w < W; ++w) mine[w] = -1;
    while (true) {
        int c = -1;                                      // lowest-index matching child of pos
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const uint64_t m = __ballot(lane + 64 * w < N && par[w] == pos && tok[w] == want);
            if (c < 0 && m != 0) c = 64 * w + __builtin_ctzll(m);
        }
        if (c < 0) break;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            if (lane + 64 * w == len) mine[w] = c;
            const int p = __shfl(pred[w], c & 63);
            if (w == (c >> 6)) want = p;
        }
        ++len;
        pos = c;
    }
    const bool fits = len <= L_max;
    if (!fits && lane == 0) flag_error(err, b, TREEWY_FLAG_BAD_PATH);
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int l = lane + 64 * w;
        if (l < L_max) path[(size_t)b * L_max + l] = fits && l < len ? mine[w] : -1;
    }
    for (int l = 64 * W + lane; l < L_max; l += 64) path[(size_t)b * L_max + l] = -1;   // past every node
    if (lane == 0) {
        path_len[b] = fits ? len : 0;
        if (bonus) bonus[b] = want;
    }
}

hipError_t launch_accept_greedy(const int32_t *parent, const int32_t *draft, const int32_t *target,
                                const int32_t *root, int N, int B, int L_max, int32_t *path,
                                int32_t *path_len, int32_t *bonus, int32_t *err, hipStream_t stream) {
    const int per_block = THREADS / 64;
    const int blocks = (B + per_block - 1) / per_block;
#define TREEWY_ACCEPT(W)                                                                                      \
    hipLaunchKernelGGL((accept_greedy_kernel<W>), dim3((unsigned)blocks), dim3(THREADS), 0, stream, parent,   \
                       draft, target, root, N, B, L_max, path, path_len, bonus, err)
    if (N <= 64) TREEWY_ACCEPT(1);
    else if (N <= 128) TREEWY_ACCEPT(2);
    else TREEWY_ACCEPT(MAX_TREE / 64);
#undef TREEWY_ACCEPT
    return hipGetLastError();
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
