// treewy_verify kernel: one workgroup (four wave64s) per (sequence, head)
// unit, launched one workgroup per unit.
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
// lane of one wave builds one row of T independently, in place over B while
// the other waves start on P (gathered into registers for shallow trees, a
// dense column sweep for deep ones).  U = T R
// and A U then run on the matrix cores with R and U taken straight from the
// accumulator registers (the contraction index is permuted to match the
// accumulator layout; T and A are read in the same permuted order).  U and
// O leave straight from their accumulators: each U store instruction writes
// whole 128-byte lines, each bf16 O store half lines, merged in L2.
//
// Streaming.  All of a unit's HBM reads are issued at once, in the order they
// are consumed (tree and gates, K/Q, V, then S0), through buffer descriptors
// bounded to the unit so padding rows read as zero without branches; two
// workgroups per CU keep HBM busy while the other one computes.  K/Q/V loads
// and U/o stores cover whole cache lines per instruction and go out
// non-temporal; S0's operand-layout loads reach each line through four
// instructions and keep the default policy so the line stays in L2 between them.
// The state written back (the fused call's S_new, the chain prefill's S_T)
// leaves in whole lines too, after a transpose across each quad of lanes.
//
// Precision.  The matrix cores take bf16; fp32 operands are split into
// hi + lo bf16 pairs and multiplied in three passes (hi*hi + hi*lo + lo*hi),
// keeping the products within ~2^-16 of fp32.  bf16 inputs are exact in bf16,
// so their products with S0 take two passes and the gram one; a bf16 state
// (SBF) is exact too, so P takes one.
//
// Variants of the same kernel (template arguments): FUSE commits the
// previous round's accepted path into S0 on the way in (the fused call) and
// writes it out as S_new; MODE walks a unit's nodes in chunks, either as a
// chain of NP-token chunks whose state is carried in registers from chunk to
// chunk and updated at the end of each (the chain prefill), or as a tree of
// more than 64 nodes in 64-node chunks, each chunk using S0 (read once and
// kept in registers) and coupled to the pseudo-values of its ancestors in
// earlier chunks before its own solve.
#include "device.h"
#include "launch.h"

namespace treewy {

// The previous round's accepted path, committed inside verify (fused call):
// S0 of this round = g_a S_old + sum_l w_l U_prev[a_l] k_prev[a_l]^T.
struct CommitArgs {
    const float *U;           // [units, N_prev, D] pseudo-values of the previous round
    const void *k;            // [units, N_prev, D] its keys, in the input dtype
    const float *alpha;       // [units, N_prev]
    const int32_t *path;      // [B, L_max] root -> accepted node
    const int32_t *path_len;  // [B]
    const int32_t *parent;    // [B, N_prev] or null (then only range and order are checked)
    void *S_new;              // [units, D, D] in the state dtype; may be S_old
    int L_max, N_prev;
    int in_stride;            // rows per unit in k and alpha (N_prev for whole tensors)
    int u_stride;             // rows per unit in U (N_prev for whole tensors)
};

template <int NP, bool F32IN, bool FUSE = false>
struct VerifyLds {
    static constexpr int XS = D + 8;                    // bf16 per staged K/Q row (pad breaks bank aliasing)
    static constexpr int MS = NP + 4;                   // floats per row of the N x N matrices
    static constexpr int X_BYTES = 2 * NP * XS * 2;     // [K; Q] in bf16
    static constexpr int XLO_OFF = X_BYTES;             // low halves of fp32 K/Q
    static constexpr int B_OFF = X_BYTES * (F32IN ? 2 : 1);
    static constexpr int M_BYTES = NP * MS * 4;
    static constexpr int A_OFF = B_OFF + M_BYTES;
    static constexpr int BETA_OFF = A_OFF + M_BYTES;
    static constexpr int G_OFF = BETA_OFF + NP * 4;     // cumulative decays: mantissas ...
    static constexpr int GE_OFF = G_OFF + NP * 4;       // ... and exponents (see DecayX)
    static constexpr int ANC_OFF = GE_OFF + NP * 4;
    static constexpr int FLAG_OFF = ANC_OFF + NP * 8;   // depth class of the chunk (see phase 3a)
    static constexpr int END = FLAG_OFF + 16;
    static constexpr int V_BYTES = NP * D * (F32IN ? 4 : 2);
    static constexpr bool V_IN_BA = V_BYTES <= 2 * M_BYTES;  // V staged over B and A before the gram
    static constexpr int V_OFF = V_IN_BA ? B_OFF : END;
    static constexpr int BASE_BYTES = V_IN_BA ? END : END + V_BYTES;
    // Chain prefill of 32-token chunks: T and A also as bf16 hi / lo planes
    // (rows of TS, columns in the kperm order of the products that read
    // them), split once by the wave that forms them instead of by every wave
    // that reads them.
    static constexpr int TS = NP + 8;                   // bf16 per plane row (16-byte aligned rows)
    static constexpr int PLANE_BYTES = NP * TS * 2;
    static constexpr int TP_OFF = BASE_BYTES;           // T hi, T lo, A hi, A lo
    static constexpr int PRE_BYTES = TP_OFF + 4 * PLANE_BYTES;
    // Fused commit: the accepted path (node, weight, then its length and g_a),
    // and CL path rows at a time, transposed: k as [d_k][CL], w U as [d_v][CL].
    static constexpr int CL = 8;
    static constexpr int META_BYTES = 64 * 4 + 64 * 4 + 16;
    static constexpr int META_OFF = BASE_BYTES;
    static constexpr int KPT_OFF = META_OFF + META_BYTES;
    static constexpr int UWT_OFF = KPT_OFF + D * CL * (F32IN ? 4 : 2);
    static constexpr int BYTES = FUSE ? UWT_OFF + D * CL * 4 : BASE_BYTES;
    // Trees of more than 64 nodes, walked in chunks of 64: every node's
    // cumulative decay (mantissa, exponent) and ancestor mask (one word per
    // chunk).  With bf16 inputs this still fits two workgroups per CU.
    static constexpr int GALL_OFF = BASE_BYTES;
    static constexpr int GEALL_OFF = GALL_OFF + MAX_TREE * 4;
    static constexpr int ANCALL_OFF = GEALL_OFF + MAX_TREE * 4;
    static constexpr int TREE_BYTES = ANCALL_OFF + MAX_TREE * MASK_WORDS * 8;
    static_assert(B_OFF % 16 == 0 && A_OFF % 16 == 0 && BETA_OFF % 16 == 0 && G_OFF % 16 == 0 && GE_OFF % 16 == 0 &&
                  ANC_OFF % 32 == 0 && V_OFF % 16 == 0 &&
                  KPT_OFF % 16 == 0 && UWT_OFF % 16 == 0 && ANCALL_OFF % 16 == 0, "alignment");
};

// One unit's HBM reads, held in registers from issue to use.  Every read goes
// through a buffer descriptor bounded to this unit's rows, so rows of padding
// nodes (t >= N) read as zero.  CHAIN: the nodes form a chain (the chain
// prefill), so there is no parent array to read.
template <int NP, bool F32IN, bool FUSE = false, bool SBF = false, bool CHAIN = false>
struct UnitReads {
    using In = typename std::conditional<F32IN, float, __bf16>::type;
    static constexpr int MT = NP / 32;
    static constexpr int CHUNK = F32IN ? 4 : 8;         // elements per 16-byte chunk
    static constexpr int CPR = D / CHUNK;               // chunks per row
    static constexpr int KQN = 2 * NP * CPR / THREADS;  // K/Q chunks per thread
    static constexpr int KN = KQN / 2;                  // the first KN are K, the rest Q
    static constexpr int ROW = D * (int)sizeof(In);     // bytes per q/k/v row
    // The wave that reads the gates and walks the tree: wave 0, except in
    // the chain prefill with 32-token chunks, where wave 2 walks each next
    // chunk while it waits for the solve (see the kernel).
    static constexpr int WALK_WAVE = CHAIN && NP == 32 ? 2 : 0;
    int par;                                            // walking wave, node = lane
    float al, be;
    uint4 kq[KQN];                                      // chunk i: row (tid / CPR + i THREADS / CPR) mod NP
    // S0 row `col`, d_k 16s + 8h + 4hg + [0, 4): four floats, or four bf16 in a uint2 for a bf16 state
    using SReg = typename std::conditional<SBF, uint2, f32x4>::type;
    static constexpr int SB = SBF ? 2 : 4;              // bytes per state entry
    SReg s0[8][2];
    static constexpr int VQN = NP * ROW / 16 / THREADS;  // V chunks per thread
    uint4 vq[VQN];                                      // V rows, 16 bytes per chunk, coalesced
    int cp_len, cp_node, cp_par;                        // fused commit, wave 1: path (lane l = entry l)
    float cp_al;                                        // and alpha_prev / parent_prev of node = lane

    // Order of the d_k index in the staged K/Q rows and in the S0 registers:
    // bits 2 and 3 swapped (an involution).  With it, contraction step s of
    // P gives lane group hg the S0 entries d_k = 16s + 4hg + [0, 4) and
    // 16s + 8 + 4hg + [0, 4), which is the row set a 32x32 accumulator tile
    // assigns to that lane group: an MFMA result over d_k lands directly in
    // these registers, and each S0 load instruction reads 32 contiguous
    // bytes of every row.
    static __device__ __forceinline__ int kperm(int j) { return (j & ~12) | ((j & 4) << 1) | ((j & 8) >> 1); }

    // Fused commit: the accepted path of unit u (lane l = entry l) with the
    // previous round's alpha and parent of node = lane.
    __device__ __forceinline__ void issue_path(const CommitArgs &cm, int u, int b, int lane) {
        const int np = cm.N_prev;
        cp_al = ld_f32(make_rsrc(cm.alpha + (size_t)u * cm.in_stride, np * 4), lane * 4);
        // (an opaque zero offset: a uniform load's result would be moved to a
        // scalar register at once, which waits for it before the unit's own reads)
        cp_len = ld_i32(make_rsrc(cm.path_len + b, 4), opaque(0));
        cp_node = ld_i32(make_rsrc(cm.path + (size_t)b * cm.L_max, cm.L_max * 4), lane * 4);
        // (without a parent array the descriptor is empty and the read gives 0:
        // no branch, so nothing here waits for these reads)
        const int32_t *pp = cm.parent;
        cp_par = ld_i32(make_rsrc(pp ? pp + (size_t)b * np : nullptr, pp ? np * 4 : 0), lane * 4);
    }

    // Every HBM read of unit u, in the order the unit consumes them.
    __device__ __forceinline__ f32x4 sget(int s, int h) const {
        if constexpr (SBF) return bf4_to_f32(s0[s][h]);
        else return s0[s][h];
    }
    __device__ __forceinline__ void sset(int s, int h, f32x4 x) {
        if constexpr (SBF) s0[s][h] = f32_to_bf4(x);
        else s0[s][h] = x;
    }

    // KQP: cache policy of the K/Q rows (tree chunks read them again).
    template <int KQP = STREAM>
    __device__ __forceinline__ void issue(const void *S0, const In *q, const In *k, const In *vv,
                                          const float *alpha, const float *beta, const int32_t *prow,
                                          int u, int N, size_t node0, bool load_state, int tid,
                                          int lane, int wave, int hg, int col) {
        if (wave == WALK_WAVE) {                        // prow: this unit's parents of the N nodes (null: a chain)
            // (read unconditionally, an empty descriptor giving 0 for a chain,
            // whose parents the walk takes as lane - 1: a branch here would
            // make the compiler wait for every outstanding memory operation.
            // The chain prefill (CHAIN) has no parent array and reads none.)
            if constexpr (!CHAIN) par = ld_i32(make_rsrc(prow, prow ? N * 4 : 0), lane * 4);
            al = ld_f32(make_rsrc(alpha + node0, N * 4), lane * 4);
            be = ld_f32(make_rsrc(beta + node0, N * 4), lane * 4);
        }

        const rsrc_t rk = make_rsrc(k + node0 * D, N * ROW), rq = make_rsrc(q + node0 * D, N * ROW);
#pragma unroll
        for (int i = 0; i < KQN; ++i) {
            const int idx = tid + THREADS * i, r = idx / CPR, c = (idx % CPR) * CHUNK;
            const int t = i < KN ? r : r - NP;
            kq[i] = ld_u32x4<KQP>(i < KN ? rk : rq, t * ROW + c * (int)sizeof(In));
        }
        const rsrc_t rv = make_rsrc(vv + node0 * D, N * ROW);
#pragma unroll
        for (int i = 0; i < VQN; ++i) vq[i] = ld_u32x4<STREAM>(rv, (tid + THREADS * i) * 16);
        // (the state's reads go last: vector reads return in order, so the
        // staging of K/Q/V then need not wait for the state.  Left to itself
        // the scheduler has moved the V reads behind them.)
        __builtin_amdgcn_sched_barrier(0);
        if (load_state) issue_state(S0, u, hg, col);    // (chain prefill: the state is already in registers)
    }

    // Writes line L (128 bytes) of each of this wave's 32 state rows to rn in
    // whole lines: the steps s of line L (two for fp32, four for bf16) hold
    // it as 16- or 8-byte pieces spread over the lanes of each quad and the
    // two lane groups.  A bf16 state first swaps pieces across the lane
    // groups so that lane group hg holds the 16-byte pieces of h = hg; then
    // a 4 x 4 transpose across each quad gives store instruction r row r of
    // every quad: eight whole lines per instruction, non-temporal.  The
    // registers read are left unchanged.
    static constexpr int LINE_STEPS = SBF ? 4 : 2;
    __device__ __forceinline__ void store_state_line(rsrc_t rn, int L, int wave, int lane) const {
        const int l32 = lane & 31, hg = lane >> 5;
        f32x4 x4[4];
        if constexpr (SBF) {
#pragma unroll
            for (int sp = 0; sp < 4; ++sp) {
                const uint2 a = s0[4 * L + sp][0], c = s0[4 * L + sp][1];
                const auto rx = __builtin_amdgcn_permlane32_swap(a.x, c.x, false, false);
                const auto ry = __builtin_amdgcn_permlane32_swap(a.y, c.y, false, false);
                x4[sp] = __builtin_bit_cast(f32x4, make_uint4(rx[0], ry[0], rx[1], ry[1]));
            }
        } else {
            x4[0] = s0[2 * L][0];
            x4[1] = s0[2 * L][1];
            x4[2] = s0[2 * L + 1][0];
            x4[3] = s0[2 * L + 1][1];
        }
        quad_transpose(x4, lane);
        constexpr int PER16 = 16 / SB;                  // state entries per 16-byte piece
        const int off = ((wave * 32 + (l32 & ~3)) * D + 8 * PER16 * L + 2 * PER16 * (l32 & 3) + PER16 * hg) * SB;
#pragma unroll
        for (int r = 0; r < 4; ++r) st_u32x4<STREAM>(rn, off + r * D * SB, __builtin_bit_cast(uint4, x4[r]));
    }

    __device__ __forceinline__ void issue_state(const void *S0, int u, int hg, int col) {
        const rsrc_t rs = make_rsrc(static_cast<const char *>(S0) + (size_t)u * D * D * SB, D * D * SB);
        const int base = (col * D + 4 * hg) * SB;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            if constexpr (SBF) {
                s0[s][0] = ld_u32x2<CACHED>(rs, base + 32 * s);        // d_k 16s + 4hg + [0, 4)
                s0[s][1] = ld_u32x2<CACHED>(rs, base + 32 * s + 16);   // d_k 16s + 8 + 4hg + [0, 4)
            } else {
                s0[s][0] = ld_f32x4<CACHED>(rs, base + 64 * s);
                s0[s][1] = ld_f32x4<CACHED>(rs, base + 64 * s + 32);
            }
        }
    }
};

// One column of the dense sweep that builds row t of a W-row diagonal block
// of T = (I + B)^{-1} (see phase 3a), then the next column down.  Compile-time
// recursion keeps every index into r static (r stays in registers).  A
// column's row read must not be hoisted far ahead (that needs a register per
// element of B): its address passes through an empty asm that also takes the
// previous column's pivot, so rows are fetched one column ahead.
template <int I, int MS, int W>
__device__ __forceinline__ void sweep_column(float (&r)[W], const float *Bm, int t, float prev) {
    if constexpr (I >= 0) {
        const float x = I < t ? -r[I] : 0.f;            // T[t, I] (zero on and above the diagonal)
        r[I] = x;
        int base = I * MS;
        asm volatile("" : "+v"(base) : "v"(prev));
        f32x4 bi[(I + 3) / 4 > 0 ? (I + 3) / 4 : 1];
#pragma unroll
        for (int c = 0; c < (I + 3) / 4; ++c) bi[c] = *reinterpret_cast<const f32x4 *>(Bm + base + 4 * c);
#pragma unroll
        for (int c = 0; c < (I + 3) / 4; ++c)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (4 * c + e < I) r[4 * c + e] = fmaf(x, bi[c][e], r[4 * c + e]);
        sweep_column<I - 1, MS>(r, Bm, t, x);
    }
}

// How a unit's nodes are walked: in one pass (at most 64 nodes), as a chain
// in chunks of NP tokens with the state carried between chunks (chain
// prefill), or as a tree of more than 64 nodes in chunks of 64, each chunk
// using S0 (read once, held in registers) and coupled to the earlier chunks.
constexpr int ONE_PASS = 0, CHAIN_PREFILL = 1, TREE_CHUNKS = 2;

// Two workgroups per CU where 256 registers per lane suffice; fp32 inputs
// at 64 nodes need the full register file (one workgroup per CU).  The chain
// prefill keeps the state in registers from chunk to chunk and still runs
// two workgroups per CU with bf16 inputs.
template <int NP, bool F32IN, bool FUSE, bool SBF, int MODE>
__global__ __launch_bounds__(THREADS, (F32IN && NP == 64) ? 1 : 2) void verify_kernel(
    const void *S0, const void *__restrict__ q_, const void *__restrict__ k_,
    const void *__restrict__ v_, const float *__restrict__ alpha, const float *__restrict__ beta,
    const int32_t *__restrict__ parent, int N_all, int in_stride, int u_stride, int H, int units,
    void *__restrict__ o_, float *U, int32_t *__restrict__ err, CommitArgs cm) {
    using In = typename std::conditional<F32IN, float, __bf16>::type;
    static_assert(!(SBF && F32IN), "a bf16 state is paired with bf16 inputs");
    constexpr bool PRE = MODE == CHAIN_PREFILL, XT = MODE == TREE_CHUNKS;
    static_assert(!(MODE != ONE_PASS && FUSE) && !(XT && NP != 64), "chunked modes run unfused, tree chunks of 64 nodes");
    // Chain prefill chunks hold NP tokens (32 or 64); tree chunks 64 nodes.
    constexpr int CN = PRE ? NP : 64;
    using L = VerifyLds<NP, F32IN, FUSE>;
    using Reads = UnitReads<NP, F32IN, FUSE, SBF, PRE>;
    constexpr int SB = Reads::SB;
    constexpr int MT = NP / 32;                          // 32-row tiles of nodes
    constexpr int XS = L::XS, MS = L::MS;
    constexpr int CHUNK = Reads::CHUNK, CPR = Reads::CPR, KQN = Reads::KQN;

    __shared__ __attribute__((aligned(16))) unsigned char lds[XT ? L::TREE_BYTES : PRE && NP == 32 ? L::PRE_BYTES : L::BYTES];
    __bf16 *Xh = reinterpret_cast<__bf16 *>(lds);
    __bf16 *Xl = reinterpret_cast<__bf16 *>(lds + L::XLO_OFF);
    float *Bm = reinterpret_cast<float *>(lds + L::B_OFF);
    float *Am = reinterpret_cast<float *>(lds + L::A_OFF);
    // (chain prefill of 32-token chunks: T and A as bf16 planes)
    constexpr bool PLANES = PRE && NP == 32;
    __bf16 *Thi = reinterpret_cast<__bf16 *>(lds + L::TP_OFF), *Tlo = Thi + NP * L::TS;
    __bf16 *Ahi = Tlo + NP * L::TS, *Alo = Ahi + NP * L::TS;
    float *be_s = reinterpret_cast<float *>(lds + L::BETA_OFF);
    float *gm_s = reinterpret_cast<float *>(lds + L::G_OFF);  // g_t = gm_s[t] 2^ge_s[t] (DecayX)
    int *ge_s = reinterpret_cast<int *>(lds + L::GE_OFF);
    uint64_t *anc_s = reinterpret_cast<uint64_t *>(lds + L::ANC_OFF);
    int *depth_s = reinterpret_cast<int *>(lds + L::FLAG_OFF);
    float *gm_all = reinterpret_cast<float *>(lds + L::GALL_OFF);           // (tree chunks)
    int *ge_all = reinterpret_cast<int *>(lds + L::GEALL_OFF);
    uint64_t *anc_all = reinterpret_cast<uint64_t *>(lds + L::ANCALL_OFF);
    constexpr int FAST = 8;                              // ancestors a lane holds in registers
    constexpr int MED = 16;                              // ancestors a lane walks with B read one step ahead
    // fused commit staging (unused otherwise)
    constexpr int CL = L::CL;
    In *KpT = reinterpret_cast<In *>(lds + L::KPT_OFF);
    float *UwT = reinterpret_cast<float *>(lds + L::UWT_OFF);
    auto meta_node = [&](int buf) { return reinterpret_cast<int *>(lds + L::META_OFF + buf * L::META_BYTES); };
    auto meta_w = [&](int buf) { return reinterpret_cast<float *>(lds + L::META_OFF + buf * L::META_BYTES + 256); };
    auto meta_len = [&](int buf) { return reinterpret_cast<int *>(lds + L::META_OFF + buf * L::META_BYTES + 512); };
    auto meta_ga = [&](int buf) { return reinterpret_cast<float *>(lds + L::META_OFF + buf * L::META_BYTES + 516); };

    const In *q = static_cast<const In *>(q_);
    const In *k = static_cast<const In *>(k_);
    const In *v = static_cast<const In *>(v_);
    In *o = static_cast<In *>(o_);

    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    Reads rd;
    // Fused commit, one wave: check the previous round's accepted path of
    // unit uu (from rd.cp_*, lane l = entry l) as treewy_commit does, and
    // write to metadata buffer `buf` the path's nodes, the weights w_l = the
    // product of alpha over the path entries after l (suffix products across
    // lanes), the length, and g_a = the product over the whole path.  A bad
    // path commits nothing.
    auto path_meta = [&](int uu, int buf, int lane) {
        const int bb = uu / H;
        const bool len_ok = rd.cp_len >= 0 && rd.cp_len <= cm.L_max;
        const int len = len_ok ? rd.cp_len : 0;
        const int a = lane < len ? rd.cp_node : -1;
        const int before = __shfl(a, lane > 0 ? lane - 1 : 0);
        const int pa = lane == 0 ? -1 : before;
        const int src = (a >= 0 && a < 64) ? a : lane;
        const int par_a = __shfl(rd.cp_par, src);
        const float al_a = __shfl(rd.cp_al, src);
        bool bad = !len_ok;
        if (lane < len) bad = bad || a < 0 || a >= cm.N_prev || a <= pa || (cm.parent && par_a != pa);
        const bool ok = !__any(bad);
        const int len_c = ok ? len : 0;
        float x = lane < len_c ? al_a : 1.f;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const float y = __shfl_down(x, off);
            x *= lane + off < 64 ? y : 1.f;
        }
        const float after = __shfl_down(x, 1);
        meta_node(buf)[lane] = lane < len_c ? a : -1;
        meta_w(buf)[lane] = lane < len_c ? (lane + 1 < 64 ? after : 1.f) : 0.f;
        if (lane == 0) {
            *meta_len(buf) = len_c;
            *meta_ga(buf) = x;
            if (!ok) flag_error(err, bb, TREEWY_FLAG_BAD_PATH);
        }
    };
    // One workgroup per unit (the launch is one workgroup per unit).
    const int u = blockIdx.x;
    if (u >= units) return;                              // (uniform across the workgroup)
    constexpr int buf = 0;                               // the fused call's path metadata buffer
    {
        const int b = u / H;
        // Chunked modes: the unit's nodes in chunks of CN (the chain prefill
        // keeps the state in registers from one chunk to the next).
        // Otherwise one pass.
        const int chunks = MODE != ONE_PASS ? (N_all + CN - 1) / CN : 1;
        // A chain's cumulative decays over its n tokens from the gates in
        // rd.al: node t's ancestors are 0 .. t - 1, and pointer jumping is
        // the inclusive prefix product below (the same factors combined in
        // the same order), one shuffle pair per stride.
        auto chain_decays = [&](int n, float &pm, int &pe) {
            const int ln = threadIdx.x & 63;
            pm = ln < n ? DecayX::mant(rd.al) : 0.f;
            pe = ln < n ? DecayX::expo(rd.al) : 0;
#pragma unroll
            for (int off = 1; off < NP; off <<= 1) {
                const float ym = __shfl_up(pm, off);
                const int ye = __shfl_up(pe, off);
                if (ln >= off && ln < n) DecayX::mul(pm, pe, ym, ye);
            }
        };
        // 32-token chunks: wave 2 walks chunk c + 1 during chunk c, in phase
        // 3, where it would wait for the solve, instead of wave 0 walking
        // each chunk at its start while the other waves wait at the staging
        // barrier.
        constexpr bool WALK_AHEAD = PRE && Reads::WALK_WAVE == 2;
        float next_pm = 0.f;
        int next_pe = 0;
        for (int chunk = 0; chunk < chunks; ++chunk) {
        // Lane indices are re-derived each pass from an opaque copy so the
        // per-lane offsets below are recomputed here instead of being hoisted
        // out of the loops and held in registers for their whole length (they
        // are re-derived again before phase 5).
        int tid = opaque(threadIdx.x), lane = tid & 63;
        int l32 = lane & 31, hg = lane >> 5;
        int col = wave * 32 + l32;                       // this lane's d_v column (= row of S0)
        const int N = MODE != ONE_PASS ? (N_all - CN * chunk < CN ? N_all - CN * chunk : CN) : N_all;
        const int base = XT ? 64 * chunk : 0;            // tree index of this chunk's node 0
        const int32_t *prow = parent ? parent + (size_t)b * N_all + base : nullptr;
        const size_t node0 = (size_t)u * in_stride + CN * chunk;   // row of node 0 in q/k/v/alpha/beta/o
        const size_t unode0 = (size_t)u * u_stride;      // ... and in U

        // Fused commit, per thread: one k chunk (KCH elements of d_k) and one
        // U chunk (4 of d_v) of the CL path rows staged per pass.
        // Fused commit, per thread: column sc of the path rows (d_k of k, d_v
        // of U) at path entries 4 sh .. 4 sh + 3 of the CL staged per pass,
        // loaded one entry at a time (a wave's 64 columns of one row per
        // instruction) and stored as one contiguous piece of the transposed
        // row, so that a wave's store covers distinct banks.
        static_assert(THREADS == 2 * D && CL == 8, "two 4-entry halves of every column");
        const int sc = tid % D, sh = tid / D;
        constexpr int OOB = 1 << 30;                     // past every descriptor: reads zero
        const rsrc_t rkp = make_rsrc(FUSE ? static_cast<const In *>(cm.k) + (size_t)u * cm.in_stride * D : nullptr,
                                     FUSE ? cm.N_prev * D * (int)sizeof(In) : 0);
        const rsrc_t rup = make_rsrc(FUSE ? cm.U + (size_t)u * cm.u_stride * D : nullptr,
                                     FUSE ? cm.N_prev * D * 4 : 0);
        const int *c_node = meta_node(buf);
        const float *c_w = meta_w(buf);
        // Entries past the path read as zero (out-of-range offset) with weight 0.
        struct PathPiece {
            In k[4];
            float u[4];
        };
        auto stage_load = [&](int l0, int clen, PathPiece &pp) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int l = l0 + 4 * sh + i;
                const int a = l < clen ? c_node[l] : -1;
                pp.k[i] = ld_elem<In>(rkp, a >= 0 ? (a * D + sc) * (int)sizeof(In) : OOB);
                pp.u[i] = ld_f32(rup, a >= 0 ? (a * D + sc) * 4 : OOB);
            }
        };
        auto stage_store = [&](int l0, const PathPiece &pp) {
            In kx[4];
            float ux[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                kx[i] = pp.k[i];
                ux[i] = c_w[l0 + 4 * sh + i] * pp.u[i];  // 0 past the path
            }
            if constexpr (F32IN)
                *reinterpret_cast<f32x4 *>(KpT + sc * CL + 4 * sh) = *reinterpret_cast<const f32x4 *>(kx);
            else
                *reinterpret_cast<bf16x4 *>(KpT + sc * CL + 4 * sh) = *reinterpret_cast<const bf16x4 *>(kx);
            *reinterpret_cast<f32x4 *>(UwT + sc * CL + 4 * sh) = *reinterpret_cast<const f32x4 *>(ux);
        };

        // Reads, in the order they are needed.  Fused: the unit's K/Q/V
        // first; then the previous round's accepted path, which wave 3 turns
        // into metadata; then every thread's share of its first CL path rows;
        // S_old last.  Vector-memory counters retire in order, so the wait for
        // the path rows (phase 1) covers K/Q/V, which staging needs anyway,
        // but not S_old, which only P needs.
        int clen = 0;
        float ga = 1.f;
        PathPiece cp;
        // The chain prefill fetches the next chunk early where the registers
        // allow: fp32 tokens (one workgroup per CU) and 32-token chunks.
        constexpr bool AHEAD = PRE && (F32IN || NP == 32);
        static_assert(!WALK_AHEAD || AHEAD, "the next chunk's gates are fetched during this one");
        // The chunked modes read S0 with the first chunk only and keep it in
        // registers (tree chunks use it unchanged in every chunk).
        if constexpr (FUSE) {
            rd.template issue<STREAM>(S0, q, k, v, alpha, beta, prow, u, N, node0, false, tid, lane, wave, hg, col);
            if (wave == 3) {
                rd.issue_path(cm, u, b, lane);
                path_meta(u, buf, lane);
            }
            __syncthreads();                             // the path metadata, from wave 3
            clen = *meta_len(buf);
            ga = *meta_ga(buf);
            stage_load(0, clen, cp);
            rd.issue_state(S0, u, hg, col);
        } else if (!AHEAD || chunk == 0) {               // (then later chunks were fetched one chunk ahead)
            rd.template issue<XT ? CACHED : STREAM>(S0, q, k, v, alpha, beta, prow, u, N, node0,
                                                    chunk == 0, tid, lane, wave, hg, col);
        }

        // ---- phase 1: ancestors and cumulative decay by pointer jumping ----
        // Lane t of the walking wave keeps (ptr, prod, mask): ptr an ancestor of t (or
        // -1), prod the product of alpha over the path (ptr, t] (in extended
        // range, DecayX: mantissa pm, exponent pe), mask the ancestors of t
        // strictly below t down to and including ptr.  Each round doubles the
        // covered path by reading the state of lane ptr, so depth d needs
        // ceil(log2 d) rounds; then prod = g_t, mask = ancestors.
        // Tree chunks: a parent in an earlier chunk already has its final
        // decay and ancestors (gm_all / ge_all, anc_all), so the lane takes
        // them over at once; ext holds the ancestor words of the earlier chunks.
        if (wave == Reads::WALK_WAVE) {
            float pm;
            int pe;
            uint64_t ext[XT ? MASK_WORDS : 1] = {};
            uint64_t mask;
            if constexpr (PRE) {
                if (WALK_AHEAD && chunk > 0) {          // walked during the previous chunk
                    pm = next_pm;
                    pe = next_pe;
                } else {
                    chain_decays(N, pm, pe);
                }
                mask = lane < N ? (1ull << lane) - 1ull : 0ull;
            } else {
            pm = lane < N ? DecayX::mant(rd.al) : 0.f;
            pe = lane < N ? DecayX::expo(rd.al) : 0;
            int ptr = lane < N ? (parent ? rd.par : lane - 1) : -1;   // (no parent array: a chain)
            if (lane < N && (ptr < -1 || ptr >= base + lane)) {
                flag_error(err, b, TREEWY_FLAG_BAD_PARENT);
                ptr = -1;
            }
            if constexpr (XT) {
                if (ptr >= 0 && ptr < base) {
                    DecayX::mul(pm, pe, gm_all[ptr], ge_all[ptr]);
#pragma unroll
                    for (int j = 0; j < MASK_WORDS; ++j)
                        ext[j] = anc_all[ptr * MASK_WORDS + j] | (j == (ptr >> 6) ? 1ull << (ptr & 63) : 0ull);
                    ptr = -1;
                } else if (ptr >= 0) {
                    ptr -= base;
                }
            }
            mask = ptr >= 0 ? (1ull << ptr) : 0ull;
            while (__any(ptr >= 0)) {
                const int src = ptr >= 0 ? ptr : lane;
                const float pm_s = __shfl(pm, src);
                const int pe_s = __shfl(pe, src);
                const int ptr_s = __shfl(ptr, src);
                const uint64_t mask_s = __shfl(mask, src);
                uint64_t ext_s[XT ? MASK_WORDS : 1] = {};
                if constexpr (XT)                        // (the words of this and later chunks are zero)
#pragma unroll
                    for (int j = 0; j < MASK_WORDS; ++j)
                        if (j < chunk) ext_s[j] = __shfl(ext[j], src);
                if (ptr >= 0) {
                    DecayX::mul(pm, pe, pm_s, pe_s);
                    mask |= mask_s;
                    ptr = ptr_s;
                    if constexpr (XT)
#pragma unroll
                        for (int j = 0; j < MASK_WORDS; ++j) ext[j] |= ext_s[j];
                }
            }
            }
            if (lane < NP) {
                gm_s[lane] = pm;
                ge_s[lane] = pe;
                be_s[lane] = lane < N ? rd.be : 0.f;
                anc_s[lane] = mask;
            }
            if constexpr (XT) {                          // base + lane < MAX_TREE: at most 4 chunks
                gm_all[base + lane] = pm;
                ge_all[base + lane] = pe;
#pragma unroll
                for (int j = 0; j < MASK_WORDS; ++j) anc_all[(base + lane) * MASK_WORDS + j] = j == chunk ? mask : ext[j];
            }
            const int depth_class = !__any(__popcll(mask) > FAST) ? 1 : !__any(__popcll(mask) > MED) ? 2 : 0;
            if (lane == 0) *depth_s = depth_class;
        }
        // Fused: the path rows go to LDS.
        if constexpr (FUSE) stage_store(0, cp);
        // K and Q into LDS as bf16 (hi/lo for fp32 input), padding rows zero,
        // with the d_k order permuted by kperm (see UnitReads::kperm).
        auto stage_x = [&](__bf16 *xh, __bf16 *xl, int r, int c, const uint4 &val) {
            if constexpr (!F32IN) {
                *reinterpret_cast<uint2 *>(xh + r * XS + Reads::kperm(c)) = make_uint2(val.x, val.y);
                *reinterpret_cast<uint2 *>(xh + r * XS + Reads::kperm(c + 4)) = make_uint2(val.z, val.w);
            } else {
                const f32x4 f = *reinterpret_cast<const f32x4 *>(&val);
                uint2 hi, lo;
                hi.x = pack_bf2(f[0], f[1]);
                hi.y = pack_bf2(f[2], f[3]);
                lo.x = pack_bf2(f[0] - __builtin_bit_cast(float, hi.x << 16),
                                f[1] - __builtin_bit_cast(float, hi.x & 0xffff0000u));
                lo.y = pack_bf2(f[2] - __builtin_bit_cast(float, hi.y << 16),
                                f[3] - __builtin_bit_cast(float, hi.y & 0xffff0000u));
                *reinterpret_cast<uint2 *>(xh + r * XS + Reads::kperm(c)) = hi;
                *reinterpret_cast<uint2 *>(xl + r * XS + Reads::kperm(c)) = lo;
            }
        };
#pragma unroll
        for (int i = 0; i < KQN; ++i) {
            const int idx = tid + THREADS * i, r = idx / CPR, c = (idx % CPR) * CHUNK;
            stage_x(Xh, Xl, r, c, rd.kq[i]);
        }
        // V rows into LDS as loaded (rows of padding nodes are zero).
        {
            uint4 *vs = reinterpret_cast<uint4 *>(lds + L::V_OFF);
#pragma unroll
            for (int i = 0; i < Reads::VQN; ++i) vs[tid + THREADS * i] = rd.vq[i];
        }
        __syncthreads();
        // V at the accumulator positions of P_K (bf16 held two to a register);
        // read before the gram overwrites the staging area.
        using VT = typename std::conditional<F32IN, float, bf16x2>::type;
        constexpr int VPER = F32IN ? 1 : 2;
        VT vr[MT][16 / VPER];
        {
            const In *vs = reinterpret_cast<const In *>(lds + L::V_OFF);
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const In x = vs[(32 * m + acc_row(r, hg)) * D + col];
                    if constexpr (F32IN)
                        vr[m][r] = x;
                    else
                        vr[m][r >> 1][r & 1] = x;
                }
        }
        __syncthreads();
        // Chain prefill: this chunk's reads are in LDS and registers now, so the
        // next chunk's are issued into the same registers and land during this
        // chunk's arithmetic.
        if constexpr (AHEAD) {
            if (chunk + 1 < chunks) {
                const int N1 = N_all - CN * (chunk + 1) < CN ? N_all - CN * (chunk + 1) : CN;
                rd.issue(S0, q, k, v, alpha, beta, nullptr, u, N1, node0 + CN, false, tid, lane, wave, hg, col);
            }
        }

        // ---- fused commit: S0 = g_a S_old + sum_l w_l U_prev[a_l] k_prev[a_l]^T
        // The rank-L term runs on the matrix cores as (K_path^T)(w U_path)
        // over 32-row blocks of d_k; its accumulator rows are exactly the d_k
        // entries this lane holds of S0 (see UnitReads::kperm), so the update
        // is elementwise.  Lane group 1 feeds zeros (CL = 8 of the 16
        // contraction slots are used).  Paths of at most CL nodes (the usual
        // case) update and store S0 block by block inside the P loop below,
        // as its pieces arrive; longer paths accumulate every CL-row pass
        // first.
        auto rank_block = [&](int jb, f32x16 acc) {     // acc += block jb of (K_path^T)(w U_path)
            const bf16x8 zero8 = {};
            float uw8[8];
            *reinterpret_cast<f32x4 *>(uw8) = *reinterpret_cast<const f32x4 *>(UwT + col * CL);
            *reinterpret_cast<f32x4 *>(uw8 + 4) = *reinterpret_cast<const f32x4 *>(UwT + col * CL + 4);
            bf16x8 ubh, ubl;
            split8(uw8, ubh, ubl);
            ubh = hg ? zero8 : ubh;
            ubl = hg ? zero8 : ubl;
            const In *krow = KpT + (32 * jb + l32) * CL;
            if constexpr (F32IN) {
                float k8[8];
                *reinterpret_cast<f32x4 *>(k8) = *reinterpret_cast<const f32x4 *>(krow);
                *reinterpret_cast<f32x4 *>(k8 + 4) = *reinterpret_cast<const f32x4 *>(krow + 4);
                bf16x8 ah, alo;
                split8(k8, ah, alo);
                acc = mma(ah, ubh, acc);
                acc = mma(ah, ubl, acc);
                acc = mma(alo, ubh, acc);
            } else {
                const bf16x8 ah = *reinterpret_cast<const bf16x8 *>(krow);
                acc = mma(ah, ubh, acc);
                acc = mma(ah, ubl, acc);
            }
            return acc;
        };
        const bool upd_in_p = FUSE && clen > 0 && clen <= CL;
        const rsrc_t rn = make_rsrc(FUSE ? static_cast<char *>(cm.S_new) + (size_t)u * D * D * SB : nullptr,
                                    FUSE ? D * D * SB : 0);
        // ---- P = [K; Q] S0^T for this wave's 32 columns --------------------
        // Run in phase 3, except that with 32 rows (one gram tile) waves 2 and
        // 3 run it during the gram (EARLY_P, phase 2).  The A operands (rows
        // of [K; Q] in LDS) are double-buffered one K-step ahead; the
        // scheduling barriers keep the compiler from hoisting every step's
        // operands at once.
        constexpr bool EARLY_P = NP == 32 && !FUSE;
        f32x16 accp[2 * MT];
        auto run_p = [&]() {
#pragma unroll
            for (int m = 0; m < 2 * MT; ++m) accp[m] = f32x16{};
            // (one buffer in the fused variant, whose update block needs the registers)
            constexpr int NBUF = FUSE ? 1 : 2;
            bf16x8 afr[NBUF][2 * MT], alo[NBUF][2 * MT];
            auto load_a = [&](int buf, int s) {
#pragma unroll
                for (int m = 0; m < 2 * MT; ++m) {
                    const __bf16 *arow = Xh + (32 * m + l32) * XS + 16 * s + 8 * hg;
                    afr[buf][m] = *reinterpret_cast<const bf16x8 *>(arow);
                    if constexpr (F32IN) alo[buf][m] = *reinterpret_cast<const bf16x8 *>(arow + (Xl - Xh));
                }
            };
            if (NBUF == 2) load_a(0, 0);
            // An fp32 state's operand for step s + 1 is split into hi / lo
            // bf16 during step s, so that the conversion runs beside the
            // matrix instructions instead of ahead of them (unfused: the
            // fused update changes the state right before its step).
            constexpr bool SPLIT_AHEAD = !FUSE && !SBF;
            auto split_state = [](const auto &st, int s, bf16x8 &h, bf16x8 &l) {   // (instantiated for an fp32 state only)
                float sv[8];
                *reinterpret_cast<f32x4 *>(sv) = st.s0[s][0];
                *reinterpret_cast<f32x4 *>(sv + 4) = st.s0[s][1];
                split8(sv, h, l);
            };
            bf16x8 nbh, nbl;
            // Tree chunks with an fp32 state: S0 is the same in every chunk, so
            // the first chunk keeps each step's hi / lo split in the registers
            // that held it and the later chunks read the split back.
            constexpr bool KEEP_SPLIT = XT && !SBF;
            const bool split_now = !KEEP_SPLIT || chunk == 0;   // (uniform)
            if constexpr (SPLIT_AHEAD)
                if (split_now) split_state(rd, 0, nbh, nbl);
            f32x16 dcur = {};
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                if (NBUF == 1)
                    load_a(0, s);
                else if (s < 7)
                    load_a((s + 1) & 1, s + 1);
                if constexpr (FUSE) {                    // S0 pieces of step s: commit update
                    if (upd_in_p) {
                        if ((s & 1) == 0) dcur = rank_block(s >> 1, f32x16{});
#pragma unroll
                        for (int h = 0; h < 2; ++h) {
                            f32x4 x = rd.sget(s, h);
#pragma unroll
                            for (int i = 0; i < 4; ++i) x[i] = fmaf(ga, x[i], dcur[8 * (s & 1) + 4 * h + i]);
                            rd.sset(s, h, x);                   // a bf16 state is rounded here, then used
                        }
                    }
                }
                bf16x8 bh, bl;
                if constexpr (SBF) {                     // a bf16 state is exact on the matrix cores
                    bh = __builtin_bit_cast(bf16x8, make_uint4(rd.s0[s][0].x, rd.s0[s][0].y, rd.s0[s][1].x,
                                                               rd.s0[s][1].y));
                } else if constexpr (SPLIT_AHEAD) {
                    if (split_now) {
                        bh = nbh;
                        bl = nbl;
                        if (s < 7) split_state(rd, s + 1, nbh, nbl);
                        if constexpr (KEEP_SPLIT) {
                            rd.s0[s][0] = __builtin_bit_cast(f32x4, bh);
                            rd.s0[s][1] = __builtin_bit_cast(f32x4, bl);
                        }
                    } else {
                        bh = __builtin_bit_cast(bf16x8, rd.s0[s][0]);
                        bl = __builtin_bit_cast(bf16x8, rd.s0[s][1]);
                    }
                } else {
                    split_state(rd, s, bh, bl);
                }
#pragma unroll
                for (int m = 0; m < 2 * MT; ++m) {
                    accp[m] = mma(afr[s % NBUF][m], bh, accp[m]);
                    if constexpr (!SBF) accp[m] = mma(afr[s % NBUF][m], bl, accp[m]);
                    if constexpr (F32IN) accp[m] = mma(alo[s % NBUF][m], bh, accp[m]);
                }
                // S_new leaves line by line once the steps that hold a line are done.
                if constexpr (FUSE) {
                    if (s % Reads::LINE_STEPS == Reads::LINE_STEPS - 1) rd.store_state_line(rn, s / Reads::LINE_STEPS, wave, lane);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        };

        // ---- phase 2: masked, decay-weighted gram tiles (lower triangle) --
        //   B[t,i] = beta_t (g_t/g_i) (k_t . k_i)  for i a strict ancestor of t
        //   A[t,i] = (g_t/g_i) (q_t . k_i)          for i ancestor-or-self of t
        // Every entry of B and A is written: the upper tile as zeros.
        constexpr int NPAIRS = MT * (MT + 1) / 2;
        // Tile (mt, nt) of B (with_k) and / or of A (with_q).
        auto gram_tile = [&](int mt, int nt, auto with_k, auto with_q) {
            constexpr bool WK = decltype(with_k)::value, WQ = decltype(with_q)::value;
            f32x16 gkk = {}, gqk = {};
            const __bf16 *ak_row = Xh + (32 * mt + l32) * XS + 8 * hg;
            const __bf16 *aq_row = Xh + (NP + 32 * mt + l32) * XS + 8 * hg;
            const __bf16 *bk_row = Xh + (32 * nt + l32) * XS + 8 * hg;
#pragma unroll 2
            for (int s = 0; s < 8; ++s) {
                const bf16x8 bk = *reinterpret_cast<const bf16x8 *>(bk_row + 16 * s);
                bf16x8 ak, aq;
                if constexpr (WK) ak = *reinterpret_cast<const bf16x8 *>(ak_row + 16 * s);
                if constexpr (WQ) aq = *reinterpret_cast<const bf16x8 *>(aq_row + 16 * s);
                if constexpr (WK) gkk = mma(ak, bk, gkk);
                if constexpr (WQ) gqk = mma(aq, bk, gqk);
                if constexpr (F32IN) {
                    const ptrdiff_t lo = Xl - Xh;
                    const bf16x8 bkl = *reinterpret_cast<const bf16x8 *>(bk_row + lo + 16 * s);
                    if constexpr (WK) {
                        const bf16x8 akl = *reinterpret_cast<const bf16x8 *>(ak_row + lo + 16 * s);
                        gkk = mma(ak, bkl, gkk);
                        gkk = mma(akl, bk, gkk);
                    }
                    if constexpr (WQ) {
                        const bf16x8 aql = *reinterpret_cast<const bf16x8 *>(aq_row + lo + 16 * s);
                        gqk = mma(aq, bkl, gqk);
                        gqk = mma(aql, bk, gqk);
                    }
                }
            }
            const int ci = 32 * nt + l32;
            // The accumulator rows come in runs of four consecutive nodes, so
            // their decays, betas and ancestor masks arrive as 16-byte LDS
            // broadcasts; bit ci of a mask sits in word nt of the row's u64
            // (a chain's masks are known: the ancestors of t < N are 0 .. t - 1).
            // Every read is issued before the first entry is formed.
            const float gmi = gm_s[ci];
            const int ei = ge_s[ci];
            f32x4 g4[4], b4[4];
            int4 e4[4];
            uint4 m01[4], m23[4];
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int t0 = 32 * mt + acc_row(4 * q4, hg);  // rows t0 .. t0 + 3
                g4[q4] = *reinterpret_cast<const f32x4 *>(gm_s + t0);
                e4[q4] = *reinterpret_cast<const int4 *>(ge_s + t0);
                if constexpr (!PRE) {
                    m01[q4] = *reinterpret_cast<const uint4 *>(anc_s + t0);
                    m23[q4] = *reinterpret_cast<const uint4 *>(anc_s + t0 + 2);
                }
                if constexpr (WK) b4[q4] = *reinterpret_cast<const f32x4 *>(be_s + t0);
            }
            const float inv_mi = 1.f / gmi;
            float av[16];                                // (planes: A's column ci, split below)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int t0 = 32 * mt + acc_row(4 * q4, hg);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = 4 * q4 + e, t = t0 + e;
                    bool strict;
                    if constexpr (PRE) {
                        strict = ci < t && t < N;
                    } else {
                        const uint32_t w = e == 0 ? (nt ? m01[q4].y : m01[q4].x) : e == 1 ? (nt ? m01[q4].w : m01[q4].z)
                                         : e == 2 ? (nt ? m23[q4].y : m23[q4].x) : (nt ? m23[q4].w : m23[q4].z);
                        strict = (w >> l32) & 1u;
                    }
                    const int et = e == 0 ? e4[q4].x : e == 1 ? e4[q4].y : e == 2 ? e4[q4].z : e4[q4].w;
                    // (the ratio is formed for every entry and then selected:
                    // left to the compiler, the selection became a branch per
                    // entry that waited on its own LDS read)
                    float rs = DecayX::ratio(g4[q4][e], et, inv_mi, ei);
                    asm volatile("" : "+v"(rs));
                    const float ratio = strict ? rs : (ci == t ? 1.f : 0.f);
                    if constexpr (WK) Bm[t * MS + ci] = strict ? b4[q4][e] * ratio * gkk[r] : 0.f;
                    if constexpr (WQ) {
                        if constexpr (PLANES) {
                            // (rounded to fp32 here, as stored in A elsewhere: the
                            // split below must not fuse this product into its lo)
                            av[r] = ratio * gqk[r];
                            asm("" : "+v"(av[r]));
                        }
                        else {
                            Am[t * MS + ci] = ratio * gqk[r];
                        }
                    }
                }
            }
            if constexpr (WQ && PLANES) {
                // rows t and t + 1 (accumulator entries r, r + 1) split by one
                // conversion pair, written at column kperm(ci) of both planes
                const int pc = Reads::kperm(ci);
#pragma unroll
                for (int r = 0; r < 16; r += 2) {
                    const int t = 32 * mt + acc_row(r, hg);
                    const uint32_t hb = pack_bf2(av[r], av[r + 1]);
                    const uint32_t lb = pack_bf2(av[r] - __builtin_bit_cast(float, hb << 16),
                                                 av[r + 1] - __builtin_bit_cast(float, hb & 0xffff0000u));
                    Ahi[t * L::TS + pc] = __builtin_bit_cast(__bf16, (unsigned short)hb);
                    Ahi[(t + 1) * L::TS + pc] = __builtin_bit_cast(__bf16, (unsigned short)(hb >> 16));
                    Alo[t * L::TS + pc] = __builtin_bit_cast(__bf16, (unsigned short)lb);
                    Alo[(t + 1) * L::TS + pc] = __builtin_bit_cast(__bf16, (unsigned short)(lb >> 16));
                }
            }
        };
        using Yes = std::true_type;
        using No = std::false_type;
        if constexpr (EARLY_P) {
            // One tile: its two products on waves 0 and 1; waves 2 and 3 run
            // their share of P meanwhile (wave 3 builds T after the barrier,
            // while waves 0 and 1 run theirs).
            if (wave == 0) {
                gram_tile(0, 0, Yes{}, No{});
            } else if (wave == 1) {
                gram_tile(0, 0, No{}, Yes{});
            } else {
                run_p();
            }
        } else if (wave < NPAIRS) {
            gram_tile(wave == 0 ? 0 : 1, wave == 2 ? 1 : 0, Yes{}, Yes{});
        } else if (MT == 2 && wave == 3) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int t = acc_row(r, hg);
                Bm[t * MS + 32 + l32] = 0.f;
                Am[t * MS + 32 + l32] = 0.f;
            }
        }

        __syncthreads();
        // (fused commit, long path: see rank_block)
        if (FUSE && clen > CL) {                        // long path: pass by pass, once S_old is in
            for (int l0 = 0; l0 < clen; l0 += CL) {      // uniform loop
                if (l0 > 0) {
                    __syncthreads();
                    PathPiece pp;
                    stage_load(l0, clen, pp);
                    stage_store(l0, pp);
                    __syncthreads();
                }
#pragma unroll
                for (int jb = 0; jb < 4; ++jb) {
                    const f32x16 d = rank_block(jb, f32x16{});
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        if ((r & 3) != 0) continue;             // four entries at a time
                        const int s2 = 2 * jb + (r >> 3), h = (r >> 2) & 1;
                        f32x4 x = rd.sget(s2, h);
#pragma unroll
                        for (int i = 0; i < 4; ++i) x[i] = l0 == 0 ? fmaf(ga, x[i], d[r + i]) : x[i] + d[r + i];
                        rd.sset(s2, h, x);
                    }
                }
            }
        }
        const int depth_class = *depth_s;
        const bool shallow = depth_class == 1, medium = depth_class == 2;
        // ---- phase 3a: rows of T = (I + B)^{-1}, on wave 3 while the others run P
        // (T (I + B))[t, j] = 0 for j != t gives, walking t's ancestors j from
        // the nearest upwards, T[t, j] = -sum over i in {t} and the ancestors
        // of t below j of T[t, i] B[i, j], with T[t, t] = 1.  Each lane
        // builds its own row t, which overwrites row t of B.
        // Shallow trees (at most FAST ancestors per node): T has the sparsity
        // of B plus the diagonal; a lane gathers the entries among its
        // ancestors into registers first.
        if (shallow && wave == 3 && lane < NP) {
            const int t = lane;
            const uint64_t anc = anc_s[t];              // (zero past the last node)
            int a[FAST];                                 // a[0] = parent(t), a[1] = its parent, ...
            uint64_t rem = anc;
#pragma unroll
            for (int kk = 0; kk < FAST; ++kk) {
                a[kk] = rem ? 63 - __builtin_clzll(rem) : t;
                rem &= ~(1ull << (a[kk] & 63));
            }
            // Past the m ancestors, a[kk] = t: those reads fetch B[t, t] and
            // B[a[l], t] (a[l] < t), which are zero, so every read is made
            // unconditionally (conditional reads became a branch and a wait
            // each) and the x past m come out zero.
            float bt[FAST], bb[FAST][FAST], x[FAST];
#pragma unroll
            for (int kk = 0; kk < FAST; ++kk) {
                bt[kk] = Bm[t * MS + a[kk]];
#pragma unroll
                for (int l = 0; l < kk; ++l) bb[l][kk] = Bm[a[l] * MS + a[kk]];
            }
#pragma unroll
            for (int kk = 0; kk < FAST; ++kk) {
                float acc = bt[kk];
#pragma unroll
                for (int l = 0; l < kk; ++l) acc += x[l] * bb[l][kk];
                x[kk] = -acc;
            }
            // (every read of B above precedes these stores)
            float *Tt = Bm + t * MS;
#pragma unroll
            for (int kk = 0; kk < FAST; ++kk) Tt[a[kk]] = x[kk];   // past m: a zero on the diagonal
            if (t < N) Tt[t] = 1.f;
        }
        // Trees of at most MED ancestors per node: the same recurrence, with
        // the entries of B that ancestor kk needs (B[t, a_kk] and B[a_l, a_kk]
        // for the nearer ancestors l) read one ancestor ahead, as too many to
        // hold at once.  The reads for ancestor kk + 1 take their column
        // offset through an empty asm that also takes x[kk - 1], so they are
        // issued while x[kk] is formed and not hoisted further.
        if (medium && wave == 3 && lane < NP) {
            const int t = lane;
            uint64_t rem = anc_s[t];
            int a[MED];
#pragma unroll
            for (int kk = 0; kk < MED; ++kk) {
                a[kk] = rem ? 63 - __builtin_clzll(rem) : t;
                rem &= ~(1ull << (a[kk] & 63));
            }
            float x[MED], cur[MED], nxt[MED];
            cur[0] = Bm[t * MS + a[0]];
#pragma unroll
            for (int kk = 0; kk < MED; ++kk) {
                if (kk + 1 < MED) {
                    int ak = a[kk + 1];
                    if (kk > 0) asm volatile("" : "+v"(ak) : "v"(x[kk - 1]));
                    nxt[0] = Bm[t * MS + ak];
#pragma unroll
                    for (int l = 0; l <= kk; ++l) nxt[l + 1] = Bm[a[l] * MS + ak];
                }
                float acc = cur[0];
#pragma unroll
                for (int l = 0; l < kk; ++l) acc += x[l] * cur[l + 1];
                x[kk] = -acc;
#pragma unroll
                for (int l = 0; l <= kk + 1 && l < MED; ++l) cur[l] = nxt[l];
            }
            // (every read of B above precedes these stores)
            float *Tt = Bm + t * MS;
#pragma unroll
            for (int kk = 0; kk < MED; ++kk) Tt[a[kk]] = x[kk];     // past m: a zero on the diagonal
            if (t < N) Tt[t] = 1.f;
        }
        // Deeper trees: the same recurrence as a dense column sweep.  Lane t
        // keeps r[j] = sum over the finished columns i of T[t, i] B[i, j]; at
        // column i (from the last down) T[t, i] = -r[i] is final and row i
        // of B (one broadcast read) is added in.  B is zero off the ancestor
        // pattern, so the sweep reaches the same T for any tree; it costs
        // n^2 / 2 fused multiply-adds per lane and no dependent LDS reads.
        // Every read of B precedes the final row stores.  With 64 rows, T is
        // built in 32 x 32 blocks on the same wave: both diagonal blocks
        // (T00 = inverse of I + B00 on lanes 0-31, T11 = inverse of I + B11
        // on lanes 32-63) in one sweep, then T10 = -T11 (B10 T00) on the
        // matrix cores, in place over B10 (M = B10 T00 is parked there first
        // so that one accumulator tile is live at a time).  LDS accesses of
        // one wave complete in order, so no barrier separates the steps.
        if (depth_class == 0 && wave == 3) {
            // (the solve, then at 64 rows this wave's share of P, is the
            // critical path here: the wave goes first at instruction issue on
            // its SIMD until then)
            __builtin_amdgcn_s_setprio(2);
            // Diagonal 16-row blocks first: lanes 16 q .. 16 q + 15 sweep T_q =
            // (I + B_qq)^{-1} in 15 column steps (two distinct broadcast
            // addresses per half-wave read; at 32 rows lanes 32-63 repeat
            // block 0 and store nothing).
            const int q = lane >> 4, tl = lane & 15;
            const bool live = 16 * q < NP;
            const int off = live ? 16 * q : 0;
            const float *Bblk = Bm + off * MS + off;
            float r[16];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const f32x4 bt = *reinterpret_cast<const f32x4 *>(Bblk + tl * MS + 4 * c);
#pragma unroll
                for (int e = 0; e < 4; ++e) r[4 * c + e] = bt[e];
            }
            sweep_column<15, MS>(r, Bblk, tl, 0.f);
            if (live) {
                float *Tt = Bm + (off + tl) * MS + off;
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    *reinterpret_cast<f32x4 *>(Tt + 4 * c) = f32x4{r[4 * c], r[4 * c + 1], r[4 * c + 2], r[4 * c + 3]};
                if (off + tl < N) Tt[tl] = 1.f;
            }
            // 32 x 32 products on the matrix cores, KS steps of 16 deep: row
            // l32 of the left factor from Arow, column l32 of the right one
            // from Bcol (rows MS apart).
            auto block_product = [&](const float *Arow, const float *Bcol, auto ks) {
                constexpr int KS = decltype(ks)::value;
                f32x16 acc = {};
#pragma unroll
                for (int s2 = 0; s2 < KS; ++s2) {
                    float a8[8], b8[8];
                    *reinterpret_cast<f32x4 *>(a8) = *reinterpret_cast<const f32x4 *>(Arow + 16 * s2 + 8 * hg);
                    *reinterpret_cast<f32x4 *>(a8 + 4) = *reinterpret_cast<const f32x4 *>(Arow + 16 * s2 + 8 * hg + 4);
#pragma unroll
                    for (int e = 0; e < 8; ++e) b8[e] = Bcol[(16 * s2 + 8 * hg + e) * MS];
                    bf16x8 ah, alo, bh, bl;
                    split8(a8, ah, alo);
                    split8(b8, bh, bl);
                    acc = mma(ah, bh, acc);
                    acc = mma(ah, bl, acc);
                    acc = mma(alo, bh, acc);
                }
                return acc;
            };
            using One = std::integral_constant<int, 1>;
            using Two = std::integral_constant<int, 2>;
            // 16 -> 32: in each 32-row diagonal block, the lower-left 16 x 16
            // block of its inverse is -T_1 (B_10 T_0), T_0 and T_1 being its
            // diagonal 16-blocks.  A 16-deep product of the block's rows with
            // its first 16 columns gives B_10 T_0 in output rows 16-31,
            // columns 0-15 (the other outputs are not used: upper entries of
            // B are zero), parked over B_10; a second, with the block's last
            // 16 columns, gives T_1 (B_10 T_0) there.
#pragma unroll
            for (int p = 0; p < NP / 32; ++p) {
                float *blk = Bm + 32 * p * MS + 32 * p;
                const f32x16 mm = block_product(blk + l32 * MS, blk + l32, One{});              // B_10 T_0
                if (l32 < 16) {
#pragma unroll
                    for (int r2 = 8; r2 < 16; ++r2) blk[acc_row(r2, hg) * MS + l32] = mm[r2];
                }
                const f32x16 tt = block_product(blk + l32 * MS + 16, blk + 16 * MS + l32, One{});  // T_1 M
                if (l32 < 16) {
#pragma unroll
                    for (int r2 = 8; r2 < 16; ++r2) blk[acc_row(r2, hg) * MS + l32] = -tt[r2];
                }
            }
            if constexpr (NP == 64) {
                // 32 -> 64: T10 = -T11 (B10 T00), with B10 T00 parked over B10
                float *B10 = Bm + 32 * MS;
                const f32x16 mm = block_product(B10 + l32 * MS, Bm + l32, Two{});            // B10 T00
#pragma unroll
                for (int r2 = 0; r2 < 16; ++r2) B10[acc_row(r2, hg) * MS + l32] = mm[r2];
                const f32x16 tt = block_product(B10 + l32 * MS + 32, B10 + l32, Two{});       // T11 M
#pragma unroll
                for (int r2 = 0; r2 < 16; ++r2) B10[acc_row(r2, hg) * MS + l32] = -tt[r2];
            }
        }

        // Chain prefill of 32-token chunks: wave 3 splits T into its bf16
        // planes once (lane: row lane % 32, columns 16 (lane / 32) .. + 15,
        // written in kperm order), after either solve has written T over B.
        if constexpr (PLANES) {
            if (wave == 3) {
                const int row = lane & 31, c0 = 16 * (lane >> 5);
                f32x4 g[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) g[c] = *reinterpret_cast<const f32x4 *>(Bm + row * MS + c0 + 4 * c);
                float x8[2][8];                          // kperm within 16 columns: groups 0, 2, then 1, 3
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    x8[0][e] = g[0][e];
                    x8[0][4 + e] = g[2][e];
                    x8[1][e] = g[1][e];
                    x8[1][4 + e] = g[3][e];
                }
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    bf16x8 th, tl;
                    split8(x8[h], th, tl);
                    *reinterpret_cast<bf16x8 *>(Thi + row * L::TS + c0 + 8 * h) = th;
                    *reinterpret_cast<bf16x8 *>(Tlo + row * L::TS + c0 + 8 * h) = tl;
                }
            }
        }

        // ---- phase 3: P (see run_p), for the waves that have not run it yet
        if (!EARLY_P || wave < 2) run_p();
        if constexpr (WALK_AHEAD) {                     // (its gates were issued with the next chunk's reads)
            if (wave == Reads::WALK_WAVE && chunk + 1 < chunks) {
                const int n1 = N_all - CN * (chunk + 1) < CN ? N_all - CN * (chunk + 1) : CN;
                chain_decays(n1, next_pm, next_pe);
            }
        }
        __builtin_amdgcn_s_setprio(0);                  // (wave 3 after a deep solve)
        __syncthreads();

        // Decays g_t of four consecutive rows t0 .. t0 + 3, as plain values.
        auto g_rows4 = [&](int t0) {
            const f32x4 m4 = *reinterpret_cast<const f32x4 *>(gm_s + t0);
            const int4 e4 = *reinterpret_cast<const int4 *>(ge_s + t0);
            return f32x4{DecayX::value(m4[0], e4.x), DecayX::value(m4[1], e4.y), DecayX::value(m4[2], e4.z),
                         DecayX::value(m4[3], e4.w)};
        };

        // ---- phase 4: R and g P_Q ---------------------------------------------
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int r4 = 0; r4 < 16; r4 += 4) {
                const int t0 = 32 * m + acc_row(r4, hg);
                const f32x4 g4 = g_rows4(t0);
                const f32x4 b4 = *reinterpret_cast<const f32x4 *>(be_s + t0);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = r4 + e;
                    float vt;
                    if constexpr (F32IN)
                        vt = vr[m][r];
                    else
                        vt = (float)vr[m][r >> 1][r & 1];
                    accp[m][r] = b4[e] * (vt - g4[e] * accp[m][r]);
                    accp[MT + m][r] *= g4[e];
                }
            }

        // ---- tree chunks: coupling to the earlier chunks ------------------
        // For t in this chunk and i in an earlier chunk j, B[t, i] U_i and
        // A[t, i] U_i enter eq. 2 through R and O, with B[t, i] =
        // beta_t (g_t / g_i) k_t . k_i and A[t, i] = (g_t / g_i) q_t . k_i
        // (i an ancestor of t).  So after phase 4 the coupling adds
        //   sum over ancestors i in chunk j of -beta_t (g_t / g_i) (k_t . k_i) U_i  to R,
        //   sum over ancestors i in chunk j of (g_t / g_i) (q_t . k_i) U_i          to O,
        // each ratio g_t / g_i <= 1 formed whole.  Per chunk j: the cross
        // gram [K; Q] K_j^T is masked and scaled into the K/Q staging area
        // (free once P is done), and its product with U_j (written by this
        // workgroup one or more chunks ago) is accumulated on the matrix
        // cores.  The chunk's own K and Q come from that staging area for the
        // first earlier chunk and from the cache after it has been
        // overwritten; K_j always from the cache.
        if constexpr (XT) {
            float *Ck = reinterpret_cast<float *>(lds), *Cq = Ck + NP * MS;
            static_assert(2 * NP * MS * 4 <= L::B_OFF, "the coupling blocks fit where K/Q were staged");
            for (int j = 0; j < chunk; ++j) {            // uniform loop
                // Chunk j's nodes with a descendant in this chunk, one bit each
                // (past the chunk's last node the ancestor words are zero).  In
                // DFS order these are the ancestors of this chunk's first node,
                // at most its depth.  The coupling runs over those columns only,
                // gathered, 32 at a time: usually one group, so half the cross
                // gram, the U_j reads and the product of all 64 columns, and
                // none of chunk j's other rows read again.
                const uint64_t need = wave_or64(anc_all[(base + lane) * MASK_WORDS + j]);
                const int nneed = __popcll(need);
                const int my_node = compact_bits(need, lane);   // lane c < nneed: node of chunk j in slot c
                const int kind = wave & 1, mt = wave >> 1;       // wave: (K or Q rows) x (32-row tile)
                constexpr int OOB = 1 << 30;                     // past every descriptor: reads zero
                const size_t row0 = (size_t)u * in_stride;
                const rsrc_t ra = make_rsrc((kind ? q : k) + (row0 + base) * D, N * Reads::ROW);
                const rsrc_t rbk = make_rsrc(k + (row0 + 64 * j) * D, 64 * Reads::ROW);
                const rsrc_t ruj = make_rsrc(U + ((size_t)u * u_stride + 64 * j) * D, 64 * D * 4);
                for (int g0 = 0; g0 < nneed; g0 += 32) {          // uniform loop
                    // (lane indices re-derived inside the loop: offsets formed
                    // from them stay in it instead of being hoisted, and held,
                    // across the coupling)
                    const int lane = opaque(threadIdx.x) & 63, l32 = lane & 31, hg = lane >> 5, col = wave * 32 + l32;
                    const int node_c = __shfl(my_node, g0 + l32);   // this lane's column
                    const bool live_c = g0 + l32 < nneed;
                    const int arow = (32 * mt + l32) * Reads::ROW, brow = live_c ? node_c * Reads::ROW : OOB;
                    f32x16 gx = {};
                    if (j == 0 && g0 == 0) {
                        // This chunk's K or Q still staged in LDS (kperm order
                        // of d_k): read it there, and chunk 0's rows in the
                        // same order, element e of step s being d_k = 16 s +
                        // 8 (e / 4) + 4 hg + e % 4.
                        const __bf16 *xa = Xh + ((kind ? NP : 0) + 32 * mt + l32) * XS + 8 * hg;
                        constexpr int XU = SBF ? 2 : 4;  // steps in flight (a bf16 state has fewer registers to spare)
#pragma unroll XU
                        for (int s = 0; s < 8; ++s) {
                            const int o0 = (16 * s + 4 * hg) * (int)sizeof(In), o1 = o0 + 8 * (int)sizeof(In);
                            const bf16x8 ah = *reinterpret_cast<const bf16x8 *>(xa + 16 * s);
                            if constexpr (F32IN) {
                                const bf16x8 al = *reinterpret_cast<const bf16x8 *>(xa + 16 * s + (Xl - Xh));
                                float x8[8];
                                *reinterpret_cast<f32x4 *>(x8) = ld_f32x4<CACHED>(rbk, brow + o0);
                                *reinterpret_cast<f32x4 *>(x8 + 4) = ld_f32x4<CACHED>(rbk, brow + o1);
                                bf16x8 bh, bl;
                                split8(x8, bh, bl);
                                gx = mma(ah, bh, gx);
                                gx = mma(ah, bl, gx);
                                gx = mma(al, bh, gx);
                            } else {
                                const uint2 b0 = ld_u32x2<CACHED>(rbk, brow + o0), b1 = ld_u32x2<CACHED>(rbk, brow + o1);
                                gx = mma(ah, __builtin_bit_cast(bf16x8, make_uint4(b0.x, b0.y, b1.x, b1.y)), gx);
                            }
                        }
                    } else {
                        // (this chunk's rows from the cache: the staging area
                        // holds the coupling blocks by now)
#pragma unroll 2
                        for (int s = 0; s < 8; ++s) {
                            const int off = (16 * s + 8 * hg) * (int)sizeof(In);
                            if constexpr (F32IN) {
                                float xa8[8], xb8[8];
                                *reinterpret_cast<f32x4 *>(xa8) = ld_f32x4<CACHED>(ra, arow + off);
                                *reinterpret_cast<f32x4 *>(xa8 + 4) = ld_f32x4<CACHED>(ra, arow + off + 16);
                                *reinterpret_cast<f32x4 *>(xb8) = ld_f32x4<CACHED>(rbk, brow + off);
                                *reinterpret_cast<f32x4 *>(xb8 + 4) = ld_f32x4<CACHED>(rbk, brow + off + 16);
                                bf16x8 ah, al, bh, bl;
                                split8(xa8, ah, al);
                                split8(xb8, bh, bl);
                                gx = mma(ah, bh, gx);
                                gx = mma(ah, bl, gx);
                                gx = mma(al, bh, gx);
                            } else {
                                const bf16x8 a8 = __builtin_bit_cast(bf16x8, ld_u32x4<CACHED>(ra, arow + off));
                                const bf16x8 b8 = __builtin_bit_cast(bf16x8, ld_u32x4<CACHED>(rbk, brow + off));
                                gx = mma(a8, b8, gx);
                            }
                        }
                    }
                    __syncthreads();                     // the coupling blocks are written over the staged K/Q (or the last group's)
                    const int ni = live_c ? node_c : 0;
                    const float inv_mi = 1.f / gm_all[64 * j + ni];  // every node of an earlier chunk is real
                    const int ei = ge_all[64 * j + ni];
                    float *Cw = kind ? Cq : Ck;
                    // (rows in runs of four, one 16-byte read of their decays
                    // each; the barrier keeps the reads from being hoisted)
#pragma unroll
                    for (int r4 = 0; r4 < 16; r4 += 4) {
                        const int t0 = 32 * mt + acc_row(r4, hg);
                        const f32x4 m4 = *reinterpret_cast<const f32x4 *>(gm_s + t0);
                        const int4 e4 = *reinterpret_cast<const int4 *>(ge_s + t0);
                        const f32x4 b4 = *reinterpret_cast<const f32x4 *>(be_s + t0);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int r = r4 + e, t = t0 + e;
                            const bool a = live_c && ((anc_all[(base + t) * MASK_WORDS + j] >> ni) & 1ull);
                            const int et = e == 0 ? e4.x : e == 1 ? e4.y : e == 2 ? e4.z : e4.w;
                            float ratio = DecayX::ratio(m4[e], et, inv_mi, ei);
                            asm volatile("" : "+v"(ratio));      // (selected below, not branched on)
                            const float val = kind ? gx[r] * ratio : -b4[e] * ratio * gx[r];
                            Cw[t * MS + l32] = a ? val : 0.f;
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
                    // This wave's columns of the gathered U_j rows, in the
                    // product's slot order.  (Issued here rather than before
                    // the barriers: each row offset takes a register of its
                    // own, and held across the epilogue they pushed the
                    // kernel past its register budget.)
                    float ub[2][8];
#pragma unroll
                    for (int s = 0; s < 2; ++s)
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int sl = g0 + 16 * s + 8 * hg + e;
                            const int nd = __shfl(my_node, sl & 63);
                            ub[s][e] = ld_f32(ruj, sl < nneed ? (nd * D + col) * 4 : OOB);
                        }
                    __syncthreads();
#pragma unroll
                    for (int s = 0; s < 2; ++s) {
                        bf16x8 bh, bl;
                        split8(ub[s], bh, bl);
#pragma unroll
                        for (int m = 0; m < 2 * MT; ++m) {
                            const float *crow = (m < MT ? Ck : Cq) + (32 * (m % MT) + l32) * MS + 16 * s + 8 * hg;
                            float c8[8];
                            *reinterpret_cast<f32x4 *>(c8) = *reinterpret_cast<const f32x4 *>(crow);
                            *reinterpret_cast<f32x4 *>(c8 + 4) = *reinterpret_cast<const f32x4 *>(crow + 4);
                            bf16x8 ah, alo;
                            split8(c8, ah, alo);
                            accp[m] = mma(ah, bh, accp[m]);
                            accp[m] = mma(ah, bl, accp[m]);
                            accp[m] = mma(alo, bh, accp[m]);
                        }
                    }
                }
                __syncthreads();                         // the coupling blocks are rewritten next (or U staged there)
            }
        }

        // Chain prefill: the Q rows staged in LDS are dead once P is done;
        // K goes there transposed for the state update at the end of the
        // chunk: row j holds K[l][d_k = j] (staged at position kperm(j)) in
        // the contraction order of that update (entry p is node l(p), the
        // accumulator row order of U), 16-byte chunks swizzled by row.
        __bf16 *KT = Xh + NP * XS, *KTl = Xl + NP * XS;
        static_assert(!PRE || D * CN * 2 <= NP * XS * 2, "K^T fits where Q was staged");
        auto kt_at = [](int j, int p) { return j * CN + (((p >> 3) ^ (j & (CN / 8 - 1))) << 3) + (p & 7); };
        if constexpr (PRE) {
            const int j = tid >> 1, p0 = (CN / 2) * (tid & 1);
#pragma unroll
            for (int c = 0; c < CN / 16; ++c) {
                bf16x8 hi, lo;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int pp = p0 + 8 * c + e, s2 = pp >> 4;
                    const int l = 32 * (s2 >> 1) + 16 * (s2 & 1) + 8 * (e >> 2) + 4 * ((pp >> 3) & 1) + (e & 3);
                    hi[e] = Xh[l * XS + Reads::kperm(j)];
                    if constexpr (F32IN) lo[e] = Xl[l * XS + Reads::kperm(j)];
                }
                *reinterpret_cast<bf16x8 *>(KT + kt_at(j, p0 + 8 * c)) = hi;
                if constexpr (F32IN) *reinterpret_cast<bf16x8 *>(KTl + kt_at(j, p0 + 8 * c)) = lo;
            }
        }
        // (no barrier: phase 4 works in registers; T was written before the
        // barrier that ends P, and the K^T writes above are read after later ones)

        // Lane indices re-derived once more for the second half of the pass,
        // so that offsets formed from them in the first half are not held in
        // registers (or spilled) across P, the solve and the coupling.
        {
            tid = opaque(threadIdx.x);
            lane = tid & 63;
            l32 = lane & 31;
            hg = lane >> 5;
            col = wave * 32 + l32;
        }
        // ---- phase 5: U = T R, then O = g P_Q + A U ------------------------
        // K-step s covers nodes [16s, 16s+16) in the order the accumulator
        // holds them: slot e of lane group hg is node 32(s/2) + 16(s%2) +
        // 8(e/4) + 4hg + e%4.
        const float *Tsrc = Bm;
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
                if (s > 2 * mt + 1) continue;            // T is zero above the diagonal blocks
                bf16x8 ah, alo;
                if constexpr (PLANES) {                  // (split once, into the planes)
                    ah = *reinterpret_cast<const bf16x8 *>(Thi + l32 * L::TS + 16 * hh + 8 * hg);
                    alo = *reinterpret_cast<const bf16x8 *>(Tlo + l32 * L::TS + 16 * hh + 8 * hg);
                } else {
                    const float *trow = Tsrc + (32 * mt + l32) * MS + 32 * m + 16 * hh + 4 * hg;
                    float ta[8];
                    *reinterpret_cast<f32x4 *>(ta) = *reinterpret_cast<const f32x4 *>(trow);
                    *reinterpret_cast<f32x4 *>(ta + 4) = *reinterpret_cast<const f32x4 *>(trow + 8);
                    split8(ta, ah, alo);
                }
                accv[mt] = mma(ah, bh, accv[mt]);
                accv[mt] = mma(ah, bl, accv[mt]);
                accv[mt] = mma(alo, bh, accv[mt]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // Chain prefill: the update weights g_N / g_l (zero past the chunk),
        // written where the ancestor masks were: those were last read before
        // the barrier that ends P, whereas beta is still read by the other
        // waves' phase 4 (no barrier orders this write after those reads).
        float *wt_s = reinterpret_cast<float *>(anc_s);
        if (PRE && wave == 0)
            wt_s[lane] = lane < N ? DecayX::ratio(gm_s[N - 1], ge_s[N - 1], 1.f / gm_s[lane], ge_s[lane]) : 0.f;
        const rsrc_t ru = make_rsrc(PRE ? nullptr : U + (unode0 + base) * D, PRE ? 0 : N * D * 4);
        const rsrc_t ro = make_rsrc(o + node0 * D, N * D * (int)sizeof(In));
        // U leaves while A U runs, straight from the accumulators (rows of
        // padding nodes fall past the end of the descriptor and are dropped):
        // each store instruction writes the lane group's 32 columns, one whole
        // 128-byte line, of two rows.  Tree chunks keep U in the cache for the
        // coupling of later chunks; the chain prefill keeps U in registers for
        // its state update and stores none.
        if constexpr (!PRE) {
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    st_f32<XT ? CACHED : STREAM>(ru, ((32 * m + acc_row(r, hg)) * D + col) * 4, accv[m][r]);
        }
#pragma unroll
        for (int s = 0; s < 2 * MT; ++s) {
            const int m = s >> 1, hh = s & 1;
            bf16x8 bh, bl;
            split8(reinterpret_cast<const float *>(&accv[m]) + 8 * hh, bh, bl);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                if (s > 2 * mt + 1) continue;
                bf16x8 ah, alo;
                if constexpr (PLANES) {                  // (split once, into the planes)
                    ah = *reinterpret_cast<const bf16x8 *>(Ahi + l32 * L::TS + 16 * hh + 8 * hg);
                    alo = *reinterpret_cast<const bf16x8 *>(Alo + l32 * L::TS + 16 * hh + 8 * hg);
                } else {
                    const float *arow = Am + (32 * mt + l32) * MS + 32 * m + 16 * hh + 4 * hg;
                    float aa[8];
                    *reinterpret_cast<f32x4 *>(aa) = *reinterpret_cast<const f32x4 *>(arow);
                    *reinterpret_cast<f32x4 *>(aa + 4) = *reinterpret_cast<const f32x4 *>(arow + 8);
                    split8(aa, ah, alo);
                }
                accp[MT + mt] = mma(ah, bh, accp[MT + mt]);
                accp[MT + mt] = mma(ah, bl, accp[MT + mt]);
                accp[MT + mt] = mma(alo, bh, accp[MT + mt]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // o straight from the accumulators as well.  With bf16 inputs a store
        // instruction writes half a line (32 bf16) of two rows; the default
        // policy lets L2 merge the halves from neighbouring waves (rows of
        // padding nodes fall past the descriptor).
        if constexpr (!F32IN) {
            // (rows r and r + 1 rounded by one conversion, stored as two halves)
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int r = 0; r < 16; r += 2) {
                    const uint32_t pr = pack_bf2(accp[MT + m][r], accp[MT + m][r + 1]);
                    __builtin_amdgcn_raw_buffer_store_b16((unsigned short)pr, ro,
                                                          ((32 * m + acc_row(r, hg)) * D + col) * 2, 0, CACHED);
                    __builtin_amdgcn_raw_buffer_store_b16((unsigned short)(pr >> 16), ro,
                                                          ((32 * m + acc_row(r + 1, hg)) * D + col) * 2, 0, CACHED);
                }
        } else {
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    st_f32<STREAM>(ro, ((32 * m + acc_row(r, hg)) * D + col) * 4, accp[MT + m][r]);
        }
        if constexpr (PRE) {
            // The chunk's state, eq. 3 over the whole chunk:
            //   S <- g_N S + sum_l (g_N / g_l) U_l k_l^T,
            // on the matrix cores as (K^T)(w U) over 32-row blocks of d_k.  The
            // B operand comes straight from the U accumulators (contraction in
            // their row order), the A operand from K^T transposed into LDS in
            // the same order; the result rows are this lane's S entries.
            __syncthreads();                             // the weights and K^T, from every wave
            const float gN = DecayX::value(gm_s[N - 1], ge_s[N - 1]);
            bf16x8 ubh[2 * MT], ubl[2 * MT];
#pragma unroll
            for (int s2 = 0; s2 < 2 * MT; ++s2) {
                float wu[8];
#pragma unroll
                for (int e4 = 0; e4 < 8; e4 += 4) {
                    const int l0 = 32 * (s2 >> 1) + acc_row(8 * (s2 & 1) + e4, hg);   // four consecutive nodes
                    const f32x4 w4 = *reinterpret_cast<const f32x4 *>(wt_s + l0);
#pragma unroll
                    for (int e = 0; e < 4; ++e) wu[e4 + e] = accv[s2 >> 1][8 * (s2 & 1) + e4 + e] * w4[e];
                }
                split8(wu, ubh[s2], ubl[s2]);
            }
#pragma unroll
            for (int jb = 0; jb < 4; ++jb) {
                const int j = 32 * jb + l32;             // d_k: row l32 of block jb of the update
                f32x16 d = {};
#pragma unroll
                for (int s2 = 0; s2 < 2 * MT; ++s2) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8 *>(KT + kt_at(j, 16 * s2 + 8 * hg));
                    d = mma(a, ubh[s2], d);
                    d = mma(a, ubl[s2], d);
                    if constexpr (F32IN) {
                        const bf16x8 alo = *reinterpret_cast<const bf16x8 *>(KTl + kt_at(j, 16 * s2 + 8 * hg));
                        d = mma(alo, ubh[s2], d);
                    }
                }
#pragma unroll
                for (int r = 0; r < 16; r += 4) {
                    const int s2 = 2 * jb + (r >> 3), h = (r >> 2) & 1;
                    f32x4 x = rd.sget(s2, h);
#pragma unroll
                    for (int i = 0; i < 4; ++i) x[i] = fmaf(gN, x[i], d[r + i]);
                    rd.sset(s2, h, x);
                }
            }
        }
        // (Tree chunks read this chunk's U rows back in later chunks: the
        // barrier makes a workgroup's global stores visible to its own later
        // loads, with no cache maintenance at workgroup scope.)
        __syncthreads();                                 // LDS is rewritten by the next chunk
        }                                                // chunk
        if constexpr (PRE) {                             // the state after the unit's last token
            const int lane = threadIdx.x & 63;
            const rsrc_t rn = make_rsrc(static_cast<char *>(cm.S_new) + (size_t)u * D * D * SB, D * D * SB);
#pragma unroll
            for (int L = 0; L < 8 / Reads::LINE_STEPS; ++L) rd.store_state_line(rn, L, wave, lane);
        }
    }
}

namespace {

template <int NP, bool F32IN, bool FUSE, bool SBF, int MODE = ONE_PASS>
hipError_t launch(const void *S0, const void *q, const void *k, const void *v, const float *alpha,
                  const float *beta, const int32_t *parent, int N, int in_stride, int u_stride, int B, int H,
                  void *o, float *U, int32_t *err, const CommitArgs &cm, hipStream_t stream) {
    // One workgroup per unit: the hardware hands each CU a new unit as soon
    // as one of its workgroups retires.  (Resident workgroups walking a fixed
    // strided list of units finished up to 13% apart, the launch waiting for
    // the slowest.)
    const int units = B * H;
    hipLaunchKernelGGL((verify_kernel<NP, F32IN, FUSE, SBF, MODE>), dim3((unsigned)units), dim3(THREADS), 0, stream,
                       S0, q, k, v, alpha, beta, parent, N, in_stride, u_stride, H, units, o, U, err, cm);
    return hipGetLastError();
}

// fp32 inputs pair with an fp32 state (the caller checks); a bf16 state with bf16 inputs.
template <bool FUSE>
hipError_t dispatch(const void *S0, const void *q, const void *k, const void *v, const float *alpha,
                    const float *beta, const int32_t *parent, int N, int in_stride, int u_stride, int B, int H,
                    bool f32_in, bool bf16_state, void *o, float *U, int32_t *err, const CommitArgs &cm,
                    hipStream_t stream) {
#define TREEWY_LAUNCH(NP, F, S)                                                                               \
    launch<NP, F, FUSE, S>(S0, q, k, v, alpha, beta, parent, N, in_stride, u_stride, B, H, o, U, err, cm, stream)
    if (bf16_state) return N <= 32 ? TREEWY_LAUNCH(32, false, true) : TREEWY_LAUNCH(64, false, true);
    if (N <= 32) return f32_in ? TREEWY_LAUNCH(32, true, false) : TREEWY_LAUNCH(32, false, false);
    return f32_in ? TREEWY_LAUNCH(64, true, false) : TREEWY_LAUNCH(64, false, false);
#undef TREEWY_LAUNCH
}

}  // namespace

hipError_t launch_verify(const void *S0, const void *q, const void *k, const void *v,
                         const float *alpha, const float *beta, const int32_t *parent, int N,
                         int B, int H, bool f32_in, bool bf16_state, void *o, float *U, int32_t *err,
                         hipStream_t stream) {
    const CommitArgs none = {};
    if (N > 64) {                                        // trees of more than 64 nodes: chunks of 64
        if (bf16_state)
            return launch<64, false, false, true, TREE_CHUNKS>(S0, q, k, v, alpha, beta, parent, N, N, N, B, H, o, U,
                                                                err, none, stream);
        if (f32_in)
            return launch<64, true, false, false, TREE_CHUNKS>(S0, q, k, v, alpha, beta, parent, N, N, N, B, H, o, U,
                                                                err, none, stream);
        return launch<64, false, false, false, TREE_CHUNKS>(S0, q, k, v, alpha, beta, parent, N, N, N, B, H, o, U,
                                                             err, none, stream);
    }
    return dispatch<false>(S0, q, k, v, alpha, beta, parent, N, N, N, B, H, f32_in, bf16_state, o, U, err, none,
                           stream);
}

hipError_t launch_commit_verify(const void *S_old, const float *U_prev, const void *k_prev,
                                const float *alpha_prev, const int32_t *path, const int32_t *path_len,
                                int L_max, const int32_t *parent_prev, int N_prev, const void *q,
                                const void *k, const void *v, const float *alpha, const float *beta,
                                const int32_t *parent, int N, int B, int H, bool f32_in, bool bf16_state,
                                void *S_new, void *o, float *U, int32_t *err, hipStream_t stream) {
    const CommitArgs cm = {U_prev, k_prev, alpha_prev, path, path_len, parent_prev, S_new, L_max, N_prev,
                           N_prev, N_prev};
    return dispatch<true>(S_old, q, k, v, alpha, beta, parent, N, N, N, B, H, f32_in, bf16_state, o, U, err, cm,
                          stream);
}

// Chain prefill: every chunk of every unit in one launch, the state kept in
// registers between chunks (see treewy_chain_prefill).  bf16 tokens run in
// 32-token chunks: the 32-row kernel has the registers to fetch the next
// chunk during the current one, and its solve is short.  fp32 tokens run in
// 64-token chunks at one workgroup per CU, also fetching ahead.
hipError_t launch_prefill(const void *S0, const void *q, const void *k, const void *v, const float *alpha,
                          const float *beta, int T, int B, int H, bool f32_in, bool bf16_state, void *S_T, void *o,
                          int32_t *err, hipStream_t stream) {
    CommitArgs cm = {};
    cm.S_new = S_T;
    if (bf16_state)
        return launch<32, false, false, true, CHAIN_PREFILL>(S0, q, k, v, alpha, beta, nullptr, T, T, 0, B, H, o, nullptr,
                                                   err, cm, stream);
    if (f32_in)
        return launch<64, true, false, false, CHAIN_PREFILL>(S0, q, k, v, alpha, beta, nullptr, T, T, 0, B, H, o, nullptr,
                                                   err, cm, stream);
    return launch<32, false, false, false, CHAIN_PREFILL>(S0, q, k, v, alpha, beta, nullptr, T, T, 0, B, H, o, nullptr, err,
                                                cm, stream);
}

}  // namespace treewy
