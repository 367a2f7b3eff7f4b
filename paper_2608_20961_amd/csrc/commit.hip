// treewy_commit kernel: rebuild the accepted node's state from the pseudo-values
// (Method, eq. 3):  S_a = g_a S0 + sum_{l} w_l U[path_l] k_{path_l}^T,
// with g_a the product of alpha along the path and w_l = g_a / g_{path_l} the
// product of alpha over the path nodes after path_l.
//
// A workgroup streams one (sequence, head) state at a time (fp32 states: the
// resident workgroups walk the units; bf16 states: one unit each): every thread owns
// sixteen 16-byte chunks at stride 4 KiB (an fp32 state: 4 entries each; a
// bf16 state: 8 entries, read and written in eight chunks), so each load and
// store instruction of the workgroup covers 4 KiB of contiguous HBM.  A bf16
// state is updated in fp32 and rounded to nearest even on the way out.  The
// path is checked one entry per thread, its weights are suffix products
// across one wave, and its scaled pseudo-value rows and keys are staged in
// LDS 64 rows at a time.  Each thread reads and writes only its own
// elements, so S_new may alias S0.
#include "device.h"
#include "launch.h"

namespace treewy {

constexpr int MAX_PATH = MAX_TREE;
constexpr int STAGE_ROWS = 64;                           // path rows staged per pass

template <bool F32K, bool SBF, bool SCALAR_PATH>
__global__ __launch_bounds__(THREADS) void commit_kernel(
    const void *S0, const float *__restrict__ U, const void *__restrict__ k_,
    const float *__restrict__ alpha, const int32_t *__restrict__ path,
    const int32_t *__restrict__ path_len, int L_max, const int32_t *__restrict__ parent, int N,
    int H, void *S_new, int32_t *__restrict__ err, int units) {
    constexpr int SB = SBF ? 2 : 4;                      // bytes per state entry
    constexpr int CH = 16 / SB;                          // entries per 16-byte chunk
    constexpr int NCH = D * D / CH / THREADS;            // chunks per thread
    using In = typename std::conditional<F32K, float, __bf16>::type;
    extern __shared__ __attribute__((aligned(16))) float stage[];   // Uw [cap][D], Kp [cap][D]
    __shared__ int s_node[MAX_PATH];
    __shared__ float s_al[MAX_PATH];
    __shared__ float s_w[MAX_PATH];
    __shared__ float s_w0;
    __shared__ int s_bad;

    const In *k = static_cast<const In *>(k_);
    const int tid = threadIdx.x;
    for (int u = blockIdx.x; u < units; u += gridDim.x) {   // resident workgroups walk the units
    const int b = u / H;
    const size_t node0 = (size_t)u * N;

    // The state is touched once: stream it past the caches on the way in and out.
    const rsrc_t rs = make_rsrc(static_cast<const char *>(S0) + (size_t)u * D * D * SB, D * D * SB);
    uint4 raw[NCH];
#pragma unroll
    for (int i = 0; i < NCH; ++i) raw[i] = ld_u32x4<STREAM>(rs, (tid + THREADS * i) * 16);

    // Entry l is valid when it lies in [0, N), follows entry l - 1 in index
    // order and (with a parent array) is its child, entry 0 a child of the
    // committed prefix.  A bad path commits nothing.
    const int len_in = path_len[b];
    bool ok = len_in >= 0 && len_in <= L_max;
    if constexpr (SCALAR_PATH) {
        // Every wave checks the whole path on wave-uniform scalar loads,
        // four entries at a time.  Those count apart from the state's vector
        // reads in flight, so the check need not wait for the state (vector
        // loads return in order).  Used where a workgroup has few units, so
        // that each unit's latency shows.
        if (ok) {
            int prev = -1;
            constexpr int PCH = 4;                       // path entries per pass (at eight, 49 scalar registers spilled)
            for (int l0 = 0; l0 < len_in; l0 += PCH) {   // uniform loop
                int a[PCH];
#pragma unroll
                for (int e = 0; e < PCH; ++e) a[e] = l0 + e < len_in ? path[(size_t)b * L_max + l0 + e] : -1;
                float al[PCH];
                int pa[PCH];
#pragma unroll
                for (int e = 0; e < PCH; ++e) {
                    const bool in_range = l0 + e < len_in && a[e] >= 0 && a[e] < N;
                    al[e] = in_range ? alpha[node0 + a[e]] : 1.f;
                    pa[e] = in_range && parent ? parent[(size_t)b * N + a[e]] : prev;
                }
#pragma unroll
                for (int e = 0; e < PCH; ++e) {
                    if (l0 + e < len_in) {
                        if (a[e] < 0 || a[e] >= N || a[e] <= prev || (parent && pa[e] != prev)) ok = false;
                        prev = a[e];
                        if (tid == e) {
                            s_node[l0 + e] = a[e];
                            s_al[l0 + e] = al[e];
                        }
                    }
                }
            }
        }
        __syncthreads();
    } else {
        // One entry per thread (the path loads wait for the state's reads,
        // which other workgroups' streams hide when a workgroup walks many
        // units).
        if (tid == 0) s_bad = ok ? 0 : 1;
        __syncthreads();
        if (ok)
            for (int l = tid; l < len_in; l += THREADS) {
                const int a = path[(size_t)b * L_max + l];
                const int prev = l > 0 ? path[(size_t)b * L_max + l - 1] : -1;
                if (a < 0 || a >= N || a <= prev || (parent && parent[(size_t)b * N + a] != prev)) {
                    s_bad = 1;
                } else {
                    s_node[l] = a;
                    s_al[l] = alpha[node0 + a];
                }
            }
        __syncthreads();
        ok = s_bad == 0;
    }
    const int len = ok ? len_in : 0;
    // w_l = product of alpha over the entries after l, and g_a = the product
    // over all: lane i of wave 0 holds entries 4i .. 4i + 3.
    if (tid < 64) {
        float a4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) a4[e] = 4 * tid + e < len ? s_al[4 * tid + e] : 1.f;
        float x = a4[0] * a4[1] * a4[2] * a4[3];
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {         // x = product over lanes >= tid
            const float y = __shfl_down(x, off);
            x *= tid + off < 64 ? y : 1.f;
        }
        const float y = __shfl_down(x, 1);
        float after = tid < 63 ? y : 1.f;                // product over the entries past this lane's four
#pragma unroll
        for (int e = 3; e >= 0; --e) {
            if (4 * tid + e < len) s_w[4 * tid + e] = after;
            after *= a4[e];
        }
        if (tid == 0) {
            s_w0 = x;
            if (!ok) flag_error(err, b, TREEWY_FLAG_BAD_PATH);
        }
    }
    __syncthreads();
    const int cap = L_max < STAGE_ROWS ? L_max : STAGE_ROWS;
    float *Uw = stage;
    float *Kp = stage + (size_t)cap * D;

    // Chunk i of this thread holds row r0 + (THREADS / (D / CH)) i, entries [c0, c0 + CH).
    const float w0 = s_w0;
    const int r0 = tid / (D / CH), c0 = (tid % (D / CH)) * CH;
    constexpr int RSTEP = THREADS / (D / CH);
    float x[NCH][CH];
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
        if constexpr (SBF) {
            const bf16x8 h = __builtin_bit_cast(bf16x8, raw[i]);
#pragma unroll
            for (int e = 0; e < CH; ++e) x[i][e] = w0 * (float)h[e];
        } else {
            const f32x4 f = __builtin_bit_cast(f32x4, raw[i]);
#pragma unroll
            for (int e = 0; e < CH; ++e) x[i][e] = w0 * f[e];
        }
    }
    for (int l0 = 0; l0 < len; l0 += cap) {             // uniform loop
        const int n = len - l0 < cap ? len - l0 : cap;
        if (l0 > 0) __syncthreads();                     // the previous pass is done with the stage
        for (int idx = tid; idx < n * D; idx += THREADS) {
            const int l = idx / D, c = idx % D;
            const size_t row = (node0 + s_node[l0 + l]) * D + c;
            Uw[idx] = s_w[l0 + l] * U[row];
            Kp[idx] = to_f32(k[row]);
        }
        __syncthreads();
        for (int l = 0; l < n; ++l) {
            float kk[CH];
#pragma unroll
            for (int e = 0; e < CH; e += 4)
                *reinterpret_cast<f32x4 *>(kk + e) = *reinterpret_cast<const f32x4 *>(Kp + l * D + c0 + e);
            const float *uw = Uw + l * D + r0;
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const float a = uw[RSTEP * i];
#pragma unroll
                for (int e = 0; e < CH; ++e) x[i][e] += a * kk[e];
            }
        }
    }
    const rsrc_t rd = make_rsrc(static_cast<char *>(S_new) + (size_t)u * D * D * SB, D * D * SB);
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
        uint4 out;
        if constexpr (SBF) {
            static_assert(CH == 8, "a bf16 state chunk is one 16-byte store");
            out = __builtin_bit_cast(uint4, round8(x[i]));
        } else {
            out = __builtin_bit_cast(uint4, f32x4{x[i][0], x[i][1], x[i][2], x[i][3]});
        }
        st_u32x4<STREAM>(rd, (tid + THREADS * i) * 16, out);
    }
    if constexpr (SBF) break;                            // a bf16 state: one unit per workgroup (see the launch)
    __syncthreads();                                     // the shared path data is rewritten by the next unit
    }                                                    // unit
}

hipError_t launch_commit(const void *S0, const float *U, const void *k, const float *alpha,
                         const int32_t *path, const int32_t *path_len, int L_max,
                         const int32_t *parent, int N, int B, int H, bool f32_k, bool bf16_state,
                         void *S_new, int32_t *err, hipStream_t stream) {
    const int units = B * H;
    const size_t lds = (size_t)2 * (L_max < STAGE_ROWS ? L_max : STAGE_ROWS) * D * sizeof(float);
    // fp32 state: a grid of resident workgroups (as many as fit on the GPU),
    // each walking units, so a workgroup starts the next unit's state reads as
    // soon as it is done.  A bf16 state (half the bytes per unit) runs faster
    // with one workgroup per unit.
    auto grid_of = [&](const void *kern) {
        if (bf16_state) return dim3((unsigned)units);
        int dev = 0, cus = 256, per_cu = 1;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, THREADS, lds) != hipSuccess || per_cu < 1)
            per_cu = 1;
        const long long g = (long long)cus * per_cu;
        return dim3((unsigned)(units < g ? units : g));
    };
    // The path check on scalar loads (see the kernel) where a workgroup has
    // at most four units; one entry per thread where it walks more.
#define TREEWY_COMMIT(F, S)                                                                                      \
    do {                                                                                                         \
        const dim3 grid = grid_of(reinterpret_cast<const void *>(&commit_kernel<F, S, false>));                  \
        if (units <= 4 * (long long)grid.x)                                                                      \
            hipLaunchKernelGGL((commit_kernel<F, S, true>), grid, dim3(THREADS), lds, stream, S0, U, k, alpha, path, \
                               path_len, L_max, parent, N, H, S_new, err, units);                                 \
        else                                                                                                     \
            hipLaunchKernelGGL((commit_kernel<F, S, false>), grid, dim3(THREADS), lds, stream, S0, U, k, alpha, path, \
                               path_len, L_max, parent, N, H, S_new, err, units);                                 \
    } while (0)
    if (f32_k) {
        if (bf16_state) TREEWY_COMMIT(true, true);
        else TREEWY_COMMIT(true, false);
    } else {
        if (bf16_state) TREEWY_COMMIT(false, true);
        else TREEWY_COMMIT(false, false);
    }
#undef TREEWY_COMMIT
    return hipGetLastError();
}

}  // namespace treewy
