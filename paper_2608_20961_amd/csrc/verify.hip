// treewy_verify kernel: one workgroup (four wave64s) per (sequence, head).
//
// The method (Method, eq. 2 and the read-out of the same solve), per unit:
//   g_t    = product of alpha over t and its ancestors
//   B[t,i] = beta_t (g_t/g_i) (k_t . k_i)          for i a strict ancestor of t, else 0
//   A[t,i] = (g_t/g_i) (q_t . k_i)                  for i ancestor-or-self of t, else 0
//   P      = [K; Q] S0^T                            (the one dense contraction)
//   R      = diag(beta) (V - diag(g) P_K)
//   U      = (I + B)^{-1} R                         (pseudo-values)
//   O      = diag(g) P_Q + A U
//
// Work split.  Wave w owns the d_v columns [32w, 32w+32) of P, R, U and O and
// the matching 32 rows of S0, which it streams from HBM straight into matrix-
// core operand registers.  K and Q are staged once in LDS as bf16 and read by
// all four waves.  T = (I + B)^{-1} has the ancestor sparsity of the tree, and
// row t of T only involves the entries of B between t's ancestors, so each
// lane of wave 0 builds one row of T independently (work ~ depth^2).  U = T R
// and A U then run on the matrix cores with R and U taken straight from the
// accumulator registers (the contraction index is permuted to match the
// accumulator layout; T and A are read in the same permuted order).
//
// Precision.  The matrix cores take bf16; fp32 operands are split into
// hi + lo bf16 pairs and multiplied in three passes (hi*hi + hi*lo + lo*hi),
// keeping the products within ~2^-16 of fp32.  bf16 inputs are exact in bf16,
// so their products with S0 take two passes and the gram one.
#include "device.h"
#include "launch.h"

namespace treewy {

template <int NP, bool F32IN>
struct VerifyLds {
    static constexpr int XS = D + 8;                    // bf16 per staged K/Q row (pad breaks bank aliasing)
    static constexpr int MS = NP + 4;                   // floats per row of the N x N matrices
    static constexpr int X_BYTES = 2 * NP * XS * 2;     // [K; Q] in bf16
    static constexpr int XLO_OFF = X_BYTES;             // low halves of fp32 K/Q
    static constexpr int B_OFF = X_BYTES * (F32IN ? 2 : 1);
    static constexpr int M_BYTES = NP * MS * 4;
    static constexpr int A_OFF = B_OFF + M_BYTES;
    static constexpr int ALPHA_OFF = A_OFF + M_BYTES;
    static constexpr int BETA_OFF = ALPHA_OFF + NP * 4;
    static constexpr int G_OFF = BETA_OFF + NP * 4;
    static constexpr int PAR_OFF = G_OFF + NP * 4;
    static constexpr int ANC_OFF = PAR_OFF + NP * 4;
    static constexpr int BYTES = ANC_OFF + NP * 8;
    static_assert(NP * MS * 4 <= X_BYTES, "T must fit where K/Q were staged");
    static_assert(B_OFF % 16 == 0 && A_OFF % 16 == 0 && ANC_OFF % 8 == 0, "alignment");
};

template <int NP, bool F32IN>
__global__ __launch_bounds__(THREADS, 2) void verify_kernel(
    const float *__restrict__ S0, const void *__restrict__ q_, const void *__restrict__ k_,
    const void *__restrict__ v_, const float *__restrict__ alpha, const float *__restrict__ beta,
    const int32_t *__restrict__ parent, int N, int H, void *__restrict__ o_, float *__restrict__ U,
    int32_t *__restrict__ err) {
    using In = typename std::conditional<F32IN, float, __bf16>::type;
    using L = VerifyLds<NP, F32IN>;
    constexpr int MT = NP / 32;                          // 32-row tiles of nodes
    constexpr int XS = L::XS, MS = L::MS;

    __shared__ __attribute__((aligned(16))) unsigned char lds[L::BYTES];
    __bf16 *Xh = reinterpret_cast<__bf16 *>(lds);
    __bf16 *Xl = reinterpret_cast<__bf16 *>(lds + L::XLO_OFF);
    float *Bm = reinterpret_cast<float *>(lds + L::B_OFF);
    float *Am = reinterpret_cast<float *>(lds + L::A_OFF);
    float *Tm = reinterpret_cast<float *>(lds);          // reuses the K/Q area once P is done
    float *al_s = reinterpret_cast<float *>(lds + L::ALPHA_OFF);
    float *be_s = reinterpret_cast<float *>(lds + L::BETA_OFF);
    float *g_s = reinterpret_cast<float *>(lds + L::G_OFF);
    int *par_s = reinterpret_cast<int *>(lds + L::PAR_OFF);
    uint64_t *anc_s = reinterpret_cast<uint64_t *>(lds + L::ANC_OFF);

    const In *q = static_cast<const In *>(q_);
    const In *k = static_cast<const In *>(k_);
    const In *v = static_cast<const In *>(v_);
    In *o = static_cast<In *>(o_);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hg = lane >> 5;
    const int u = blockIdx.x, b = u / H;
    const size_t node0 = (size_t)u * N;                  // row of node 0 of this unit in q/k/v/o/U
    const int col = wave * 32 + l32;                     // this lane's d_v column (= row of S0)

    // ---- phase 0: issue every HBM read of the unit -------------------------
    // S0 rows of this wave as matrix-core B operands: step s covers d_k [16s, 16s+16).
    f32x4 s0r[8][2];
    {
        const float *src = S0 + (size_t)u * D * D + (size_t)col * D + 8 * hg;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            s0r[s][0] = *reinterpret_cast<const f32x4 *>(src + 16 * s);
            s0r[s][1] = *reinterpret_cast<const f32x4 *>(src + 16 * s + 4);
        }
    }
    // V at the accumulator positions of P_K.
    float vr[MT][16];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int t = 32 * m + acc_row(r, hg);
            vr[m][r] = t < N ? to_f32(v[(node0 + t) * D + col]) : 0.f;
        }
    if (tid < NP) {
        const int t = tid;
        al_s[t] = t < N ? alpha[node0 + t] : 1.f;
        be_s[t] = t < N ? beta[node0 + t] : 0.f;
        par_s[t] = t < N ? parent[(size_t)b * N + t] : -1;
        g_s[t] = 0.f;
        anc_s[t] = 0;
    }
    // K rows [0, NP) and Q rows [NP, 2NP) into LDS as bf16 (hi/lo for fp32 input).
    if constexpr (!F32IN) {
        for (int idx = tid; idx < 2 * NP * 16; idx += THREADS) {
            const int r = idx >> 4, c = (idx & 15) * 8;
            const int t = r < NP ? r : r - NP;
            const In *src = r < NP ? k : q;
            uint4 val = {0u, 0u, 0u, 0u};
            if (t < N) val = *reinterpret_cast<const uint4 *>(src + (node0 + t) * D + c);
            *reinterpret_cast<uint4 *>(Xh + r * XS + c) = val;
        }
    } else {
        for (int idx = tid; idx < 2 * NP * 32; idx += THREADS) {
            const int r = idx >> 5, c = (idx & 31) * 4;
            const int t = r < NP ? r : r - NP;
            const In *src = r < NP ? k : q;
            f32x4 val = {0.f, 0.f, 0.f, 0.f};
            if (t < N) val = *reinterpret_cast<const f32x4 *>(src + (node0 + t) * D + c);
            bf16x4 hi, lo;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                hi[e] = (__bf16)val[e];
                lo[e] = (__bf16)(val[e] - (float)hi[e]);
            }
            *reinterpret_cast<bf16x4 *>(Xh + r * XS + c) = hi;
            *reinterpret_cast<bf16x4 *>(Xl + r * XS + c) = lo;
        }
    }
    {
        uint4 *z = reinterpret_cast<uint4 *>(lds + L::B_OFF);
        for (int idx = tid; idx < 2 * L::M_BYTES / 16; idx += THREADS) z[idx] = uint4{0u, 0u, 0u, 0u};
    }
    __syncthreads();

    // ---- phase 1: walk each node's ancestors (wave 0, lane t) -------------
    // Row t of Bm temporarily holds the decay ratios g_t/g_i of t's ancestors
    // (1 on the diagonal); g_t and the ancestor bit mask go to g_s / anc_s.
    if (wave == 0 && lane < N) {
        const int t = lane;
        Bm[t * MS + t] = 1.f;
        float ratio = 1.f;
        uint64_t mask = 0;
        bool bad = false;
        for (int cur = t;;) {
            ratio *= al_s[cur];
            int p = par_s[cur];
            if (p < -1 || p >= cur) {
                bad = true;
                p = -1;
            }
            if (p < 0) break;
            Bm[t * MS + p] = ratio;
            mask |= 1ull << p;
            cur = p;
        }
        g_s[t] = ratio;
        anc_s[t] = mask;
        if (bad) flag_error(err, b, TREEWY_FLAG_BAD_PARENT);
    }
    __syncthreads();

    // ---- phase 2: masked, decay-weighted gram tiles (lower triangle) ------
    constexpr int NPAIRS = MT * (MT + 1) / 2;
    if (wave < NPAIRS) {
        const int mt = wave == 0 ? 0 : 1;
        const int nt = wave == 2 ? 1 : 0;
        f32x16 gkk = {}, gqk = {};
        const __bf16 *ak_row = Xh + (32 * mt + l32) * XS + 8 * hg;
        const __bf16 *aq_row = Xh + (NP + 32 * mt + l32) * XS + 8 * hg;
        const __bf16 *bk_row = Xh + (32 * nt + l32) * XS + 8 * hg;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const bf16x8 ak = *reinterpret_cast<const bf16x8 *>(ak_row + 16 * s);
            const bf16x8 aq = *reinterpret_cast<const bf16x8 *>(aq_row + 16 * s);
            const bf16x8 bk = *reinterpret_cast<const bf16x8 *>(bk_row + 16 * s);
            gkk = mma(ak, bk, gkk);
            gqk = mma(aq, bk, gqk);
            if constexpr (F32IN) {
                const ptrdiff_t lo = Xl - Xh;
                const bf16x8 akl = *reinterpret_cast<const bf16x8 *>(ak_row + lo + 16 * s);
                const bf16x8 aql = *reinterpret_cast<const bf16x8 *>(aq_row + lo + 16 * s);
                const bf16x8 bkl = *reinterpret_cast<const bf16x8 *>(bk_row + lo + 16 * s);
                gkk = mma(ak, bkl, gkk);
                gkk = mma(akl, bk, gkk);
                gqk = mma(aq, bkl, gqk);
                gqk = mma(aql, bk, gqk);
            }
        }
        const int i = 32 * nt + l32;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int t = 32 * mt + acc_row(r, hg);
            const float dr = Bm[t * MS + i];
            Bm[t * MS + i] = i < t ? be_s[t] * dr * gkk[r] : 0.f;
            Am[t * MS + i] = dr * gqk[r];
        }
    }

    // ---- phase 3: P = [K; Q] S0^T for this wave's 32 columns --------------
    f32x16 accp[2 * MT];
#pragma unroll
    for (int m = 0; m < 2 * MT; ++m) accp[m] = f32x16{};
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        float sv[8];
        *reinterpret_cast<f32x4 *>(sv) = s0r[s][0];
        *reinterpret_cast<f32x4 *>(sv + 4) = s0r[s][1];
        bf16x8 bh, bl;
        split8(sv, bh, bl);
#pragma unroll
        for (int m = 0; m < 2 * MT; ++m) {
            const __bf16 *arow = Xh + (32 * m + l32) * XS + 16 * s + 8 * hg;
            const bf16x8 a = *reinterpret_cast<const bf16x8 *>(arow);
            accp[m] = mma(a, bh, accp[m]);
            accp[m] = mma(a, bl, accp[m]);
            if constexpr (F32IN) {
                const bf16x8 alo = *reinterpret_cast<const bf16x8 *>(arow + (Xl - Xh));
                accp[m] = mma(alo, bh, accp[m]);
            }
        }
    }
    __syncthreads();

    // ---- phase 4: rows of T = (I + B)^{-1} (wave 0); R and g P_Q (all) ----
    // (T (I + B))[t, j] = 0 for j != t gives, walking t's ancestors j from
    // the nearest upwards, T[t, j] = -sum over i in {t} and the ancestors of
    // t below j of T[t, i] B[i, j], with T[t, t] = 1.
    if (wave == 0) {
        if (lane < NP) {
            f32x4 *row = reinterpret_cast<f32x4 *>(Tm + lane * MS);
#pragma unroll
            for (int c = 0; c < MS / 4; ++c) row[c] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        if (lane < N) {
            const int t = lane;
            float *Tt = Tm + t * MS;
            Tt[t] = 1.f;
            const uint64_t anc = anc_s[t];
            uint64_t rem = anc;
            while (rem) {
                const int j = 63 - __builtin_clzll(rem);
                rem &= ~(1ull << j);
                float acc = Bm[t * MS + j];
                uint64_t below = anc & ~((2ull << j) - 1ull);   // ancestors of t deeper than j
                while (below) {
                    const int i = __builtin_ctzll(below);
                    below &= below - 1;
                    acc += Tt[i] * Bm[i * MS + j];
                }
                Tt[j] = -acc;
            }
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int t = 32 * m + acc_row(r, hg);
            const float gt = g_s[t];
            accp[m][r] = be_s[t] * (vr[m][r] - gt * accp[m][r]);
            accp[MT + m][r] *= gt;
        }
    __syncthreads();

    // ---- phase 5: U = T R, then O = g P_Q + A U ---------------------------
    // K-step s covers nodes [16s, 16s+16) in the order the accumulator holds
    // them: slot e of lane group hg is node 32(s/2) + 16(s%2) + 8(e/4) + 4hg + e%4.
    f32x16 accv[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) accv[m] = f32x16{};
#pragma unroll
    for (int s = 0; s < 2 * MT; ++s) {
        const int m = s >> 1, hh = s & 1;
        bf16x8 bh, bl;
        split8(reinterpret_cast<const float *>(&accp[m]) + 8 * hh, bh, bl);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            if (s > 2 * mt + 1) continue;                // T is zero above the diagonal blocks
            const float *trow = Tm + (32 * mt + l32) * MS + 32 * m + 16 * hh + 4 * hg;
            float ta[8];
            *reinterpret_cast<f32x4 *>(ta) = *reinterpret_cast<const f32x4 *>(trow);
            *reinterpret_cast<f32x4 *>(ta + 4) = *reinterpret_cast<const f32x4 *>(trow + 8);
            bf16x8 ah, alo;
            split8(ta, ah, alo);
            accv[mt] = mma(ah, bh, accv[mt]);
            accv[mt] = mma(ah, bl, accv[mt]);
            accv[mt] = mma(alo, bh, accv[mt]);
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int t = 32 * m + acc_row(r, hg);
            if (t < N) U[(node0 + t) * D + col] = accv[m][r];
        }
#pragma unroll
    for (int s = 0; s < 2 * MT; ++s) {
        const int m = s >> 1, hh = s & 1;
        bf16x8 bh, bl;
        split8(reinterpret_cast<const float *>(&accv[m]) + 8 * hh, bh, bl);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            if (s > 2 * mt + 1) continue;
            const float *arow = Am + (32 * mt + l32) * MS + 32 * m + 16 * hh + 4 * hg;
            float aa[8];
            *reinterpret_cast<f32x4 *>(aa) = *reinterpret_cast<const f32x4 *>(arow);
            *reinterpret_cast<f32x4 *>(aa + 4) = *reinterpret_cast<const f32x4 *>(arow + 8);
            bf16x8 ah, alo;
            split8(aa, ah, alo);
            accp[MT + mt] = mma(ah, bh, accp[MT + mt]);
            accp[MT + mt] = mma(ah, bl, accp[MT + mt]);
            accp[MT + mt] = mma(alo, bh, accp[MT + mt]);
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int t = 32 * m + acc_row(r, hg);
            if (t < N) o[(node0 + t) * D + col] = from_f32<In>(accp[MT + m][r]);
        }
}

hipError_t launch_verify(const float *S0, const void *q, const void *k, const void *v,
                         const float *alpha, const float *beta, const int32_t *parent, int N,
                         int B, int H, bool f32_in, void *o, float *U, int32_t *err,
                         hipStream_t stream) {
    const dim3 grid((unsigned)(B * H)), block(THREADS);
    if (N <= 32) {
        if (f32_in)
            hipLaunchKernelGGL((verify_kernel<32, true>), grid, block, 0, stream, S0, q, k, v, alpha,
                               beta, parent, N, H, o, U, err);
        else
            hipLaunchKernelGGL((verify_kernel<32, false>), grid, block, 0, stream, S0, q, k, v, alpha,
                               beta, parent, N, H, o, U, err);
    } else {
        if (f32_in)
            hipLaunchKernelGGL((verify_kernel<64, true>), grid, block, 0, stream, S0, q, k, v, alpha,
                               beta, parent, N, H, o, U, err);
        else
            hipLaunchKernelGGL((verify_kernel<64, false>), grid, block, 0, stream, S0, q, k, v, alpha,
                               beta, parent, N, H, o, U, err);
    }
    return hipGetLastError();
}

}  // namespace treewy
