// Fused chunkwise SFDA forward on gfx950: one workgroup per (batch, head, slice of value
// columns) scans the chunks of its sequence in order, keeping the state on chip.
//
// Method (Thm 4.2 / Cor. 4.3 chunk-WY factors, Thm 4.4 affine transfer, Thm 4.5 prefix
// outputs, eq. (apply-transfer) boundary scan).  Inside a chunk of C tokens, with
// g_t = lambda_1 * ... * lambda_t (the diagonal of Gamma_t) and S the state entering the
// chunk, unrolling the recurrence in the form S_t = Lambda_t S_{t-1} + k_t delta_t gives
//   delta_t = beta_t (v_t^* - k_t^* Lambda_t S_{t-1})
//   (I + D_beta L') Delta = D_beta (conj(V) - (conj(K) * G) S)
//   L'[t, j] = k_t^* diag(g_t / g_j) k_j  (j < t)         -- the paper's Gram-like matrix
//   O^*   = (conj(Q) * G) S + tril(A) Delta,  A[r, j] = q_r^* diag(g_r / g_j) k_j  (j <= r)
//   S_out = diag(g_C) (S + (K / G)^T Delta)
// so T = (I + D_beta L')^{-1} D_beta = D_beta M with M the paper's unit lower-triangular WY
// factor, Y = diag(g_C) (K / G)^T D_beta and W = conj(G) * K.  The state-independent part
// (g, L', A, T, T conj(V), T (conj(K) * G)) only reads this chunk's inputs; the state-
// dependent part (Delta, O, S_out) is column-separable in the value columns, so each wave
// owns a set of value columns and keeps its share of S in MFMA accumulators for the whole
// scan -- no barrier is needed between the state-dependent products.
//
// Stages per chunk (4 waves, 256 threads):
//   L  load alpha, theta (cumulative log-decay and phase), q, k, beta; write conj(Q) * G,
//      conj(K) * G and K / G to LDS (fp32); prefetch this wave's conj(V) fragments
//   G  Gram products L' (strict lower) and A (lower) on MFMA, packed in one C x C buffer
//   S  T via blocked forward substitution: 16 x 16 diagonal blocks by one lane per column,
//      off-diagonal blocks level by level on fp32 MFMA
//   W  U = T conj(V) (kept in registers), Wt = T (conj(K) * G) (to LDS)
//   D  Delta = U - Wt S, O = (conj(Q) * G) S + tril(A) Delta, S = diag(g_C)(S + (K/G)^T Delta)
//
// Numerics: g_t is formed from fp32 running sums of log alpha and theta (local to the
// chunk), so K / G grows like exp(-sum log alpha); the caller keeps the in-chunk decay
// product above ~1e-30.  Accumulation and the state are fp32; with PREC_BF16 the matrix
// products take bf16 operands (the solve always runs in fp32).
#include <type_traits>

#include "sfda_device.h"
#include "sfda_launch.h"

namespace sfda {

constexpr int MP = 64;            // key channels handled per workgroup (m is zero-padded)
constexpr int LDX = MP + 1;       // complex row stride of the C x MP operand arrays
constexpr int NTHR = 256;

struct ChunkArgs {
    const void *q, *k, *v, *alpha, *theta, *beta;
    const float* S0;
    void* o;
    float* S_T;
    int T, m, n, n_slices, slice;
    // GATED: alpha = amin + aspan sigmoid(a), theta = tmax tanh(b), beta = sigmoid(c),
    // k = k~ / (||k~|| + eps) from the pre-activations passed in alpha, theta, beta, k
    float amin, aspan, tmax, eps;
};

__device__ __forceinline__ float sigmoid_acc(float x) { return 1.f / (1.f + expf(-x)); }

template <int C>
struct ChunkSmem {
    static constexpr int LDG = C + 1;
    float2 qg[C * LDX];      // conj(q_t) * g_t
    float2 kg[C * LDX];      // conj(k_t) * g_t, later Wt = T (conj(K) * G)
    float2 ki[C * LDX];      // k_t / g_t
    float2 g2[C * LDG];      // packed: L' (strict lower) -> N; A^T (strict upper); A diag
    float beta[C];
    float2 gc[MP];           // g_C
    float sega[4][MP];
    float segp[4][MP];
};

template <int P, typename TIN, typename TOUT, int C, bool GATED>
__global__ __launch_bounds__(NTHR, 1) void chunk_kernel(ChunkArgs args)
{
    constexpr int NRB = C / 16;          // 16-token blocks per chunk
    constexpr int SEG = C / 4;           // tokens per thread in the cumulative sums
    constexpr int LDG = ChunkSmem<C>::LDG;
    constexpr int CBW = 2;               // value column blocks (8 complex columns) per wave
    __shared__ ChunkSmem<C> sm;

    const TIN* __restrict__ gq = static_cast<const TIN*>(args.q);
    const TIN* __restrict__ gk = static_cast<const TIN*>(args.k);
    const TIN* __restrict__ gv = static_cast<const TIN*>(args.v);
    const TIN* __restrict__ ga = static_cast<const TIN*>(args.alpha);
    const TIN* __restrict__ gth = static_cast<const TIN*>(args.theta);
    const TIN* __restrict__ gb = static_cast<const TIN*>(args.beta);
    TOUT* __restrict__ go = static_cast<TOUT*>(args.o);

    const int T = args.T, m = args.m, n = args.n;
    const long bh = blockIdx.x / args.n_slices;
    const int sl = blockIdx.x - static_cast<int>(bh) * args.n_slices;
    const int n0 = sl * args.slice;                       // first value column of the slice
    const int ncb = (min(args.slice, n - n0) + 7) / 8;    // active column blocks

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int c = lane & 15;          // tile row / column
    const int g = lane >> 4;          // lane group
    const int qp = lane & 1;          // part (re / im) of this lane's output column

    float* qgf = reinterpret_cast<float*>(sm.qg);
    float* kgf = reinterpret_cast<float*>(sm.kg);
    float* g2f = reinterpret_cast<float*>(sm.g2);

    const long base_tm = bh * static_cast<long>(T) * m;   // [b,h,0,0] of q, k, alpha, theta
    const long base_tn = bh * static_cast<long>(T) * n;   // [b,h,0,0] of v, o
    const long base_mn = bh * static_cast<long>(m) * n;   // [b,h,0,0] of S0, S_T

    // ---------------------------------------------------------------- state in registers
    f32x4 Sacc[CBW][MP / 16];
#pragma unroll
    for (int w = 0; w < CBW; ++w) {
        const int cb = wave + 4 * w;
        const int j = n0 + cb * 8 + (c >> 1);
#pragma unroll
        for (int kb = 0; kb < MP / 16; ++kb) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = kb * 16 + 4 * g + r;
                float x = 0.f;
                if (args.S0 != nullptr) {   // uniform branch; the load itself is unconditional
                    const bool ok = cb < ncb && j < n && i < m;
                    x = masked(ok, args.S0[2 * (base_mn + static_cast<long>(min(i, m - 1)) * n + min(j, n - 1)) + qp]);
                }
                Sacc[w][kb][r] = x;
            }
        }
    }

    const int nchunks = (T + C - 1) / C;
    for (int ch = 0; ch < nchunks; ++ch) {
        const int t0 = ch * C;

        // ============================================================ L: load, g, operands
        // this wave's conj(V) B-fragments for U = T conj(V): v[t0 + kb*16 + 4g + r][col]
        float2 vf[CBW][NRB][4];
#pragma unroll
        for (int w = 0; w < CBW; ++w) {
            const int cb = wave + 4 * w;
            const int j = n0 + cb * 8 + (c >> 1);
#pragma unroll
            for (int kb = 0; kb < NRB; ++kb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = t0 + kb * 16 + 4 * g + r;
                    const bool ok = cb < ncb && j < n && t < T;
                    float2 x = make_float2(0.f, 0.f);
                    if (gv != nullptr)      // v == NULL reads as zeros (uniform branch)
                        x = Elem<TIN>::load2(gv, base_tn + static_cast<long>(min(t, T - 1)) * n + min(j, n - 1));
                    vf[w][kb][r] = masked(ok, x);
                }
        }
        {
            const int i = tid & 63;
            const int seg = tid >> 6;
            float la[SEG], ph[SEG];
            float sa = 0.f, sp = 0.f;
#pragma unroll
            for (int u = 0; u < SEG; ++u) {
                const int t = t0 + seg * SEG + u;
                const bool ok = t < T && i < m;
                const long e = base_tm + static_cast<long>(min(t, T - 1)) * m + min(i, m - 1);
                const float a_ld = pin(Elem<TIN>::load(ga, e));
                float th = masked(ok, Elem<TIN>::load(gth, e));
                float a = ok ? a_ld : 1.f;
                if constexpr (GATED) {      // padding stays the identity token (alpha = 1, theta = 0)
                    a = ok ? args.amin + args.aspan * sigmoid_acc(a_ld) : 1.f;
                    th = ok ? args.tmax * tanhf(th) : 0.f;
                }
                sa += __logf(a);
                sp += th;
                la[u] = sa;
                ph[u] = sp;
            }
            sm.sega[seg][i] = sa;
            sm.segp[seg][i] = sp;
            {
                const int tb = t0 + (tid & (C - 1));
                float bv = Elem<TIN>::load(gb, bh * static_cast<long>(T) + min(tb, T - 1));
                if constexpr (GATED) bv = sigmoid_acc(bv);
                if (tid < C) sm.beta[tid] = masked(tb < T, bv);
            }
            __syncthreads();
            float oa = 0.f, op = 0.f;
            for (int s2 = 0; s2 < seg; ++s2) {
                oa += sm.sega[s2][i];
                op += sm.segp[s2][i];
            }
#pragma unroll
            for (int u = 0; u < SEG; ++u) {
                const int tl = seg * SEG + u;
                const int t = t0 + tl;
                const float A = la[u] + oa;
                const float Ph = ph[u] + op;
                const float e = __expf(A);
                const float ei = __expf(-A);
                float sn, cs;
                __sincosf(Ph, &sn, &cs);
                const float gr = e * cs, gi = e * sn;        // g_t
                const float hr = ei * cs, hi = -ei * sn;     // 1 / g_t
                const bool ok = t < T && i < m;
                const long e2 = base_tm + static_cast<long>(min(t, T - 1)) * m + min(i, m - 1);
                float2 qq = Elem<TIN>::load2(gq, e2), kk = Elem<TIN>::load2(gk, e2);
                qq = masked(ok, qq);
                kk = masked(ok, kk);
                if constexpr (GATED) {
                    // 1 / (||k~_t|| + eps): the wave holds channel i = lane of token t
                    float s2 = kk.x * kk.x + kk.y * kk.y;
#pragma unroll
                    for (int sh = 1; sh < 64; sh <<= 1) s2 += __shfl_xor(s2, sh);
                    const float den = sqrtf(s2) + args.eps;
                    const float inv = den > 0.f ? 1.f / den : 0.f;
                    kk.x *= inv;
                    kk.y *= inv;
                }
                sm.qg[tl * LDX + i] = make_float2(qq.x * gr + qq.y * gi, qq.x * gi - qq.y * gr);
                sm.kg[tl * LDX + i] = make_float2(kk.x * gr + kk.y * gi, kk.x * gi - kk.y * gr);
                sm.ki[tl * LDX + i] = make_float2(kk.x * hr - kk.y * hi, kk.x * hi + kk.y * hr);
                if (tl == C - 1) sm.gc[i] = make_float2(gr, gi);
            }
        }
        __syncthreads();

        // ============================================================ G: L' and A
        {
            constexpr int NCB = C / 8;                       // real column blocks of C x C
            constexpr int NT1 = NRB * (NRB + 1);             // causal tiles per matrix
            for (int tile = wave; tile < 2 * NT1; tile += 4) {
                const int mat = tile / NT1;                  // 0: L' from conj(K)G, 1: A from conj(Q)G
                int rem = tile - mat * NT1, rb = 0;
                while (rem >= min(NCB, 2 * rb + 2)) { rem -= min(NCB, 2 * rb + 2); ++rb; }
                const int cb = rem;
                const float2* X = mat ? sm.qg : sm.kg;
                const int row = rb * 16 + c;
                const int jcol = cb * 8 + (c >> 1);
                f32x4 acc = zero4();
#pragma unroll
                for (int kb = 0; kb < MP / 16; ++kb) {
                    Frag8 a, b;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int i = kb * 16 + 4 * g + r;
                        const float2 x = X[row * LDX + i];
                        a.v[2 * r] = x.x;
                        a.v[2 * r + 1] = x.y;
                        const float2 y = sm.ki[jcol * LDX + i];   // B(i, j) = (K/G)^T
                        bpair(b, r, y.x, y.y, qp);
                    }
                    mma<P>(acc, a, b);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = rb * 16 + 4 * g + r;
                    if (mat == 0) {
                        if (jcol < t) g2f[2 * (t * LDG + jcol) + qp] = acc[r];
                    } else {
                        if (jcol < t) g2f[2 * (jcol * LDG + t) + qp] = acc[r];
                        else if (jcol == t) g2f[2 * (t * LDG + t) + qp] = acc[r];
                    }
                }
            }
        }
        __syncthreads();

        // ============================================================ S: N = (I + D_beta L')^{-1}
        if (wave < NRB) {
            // diagonal block p = wave; lane jj owns column jj of N_pp
            const int p = wave;
            const int jj = lane & 15;
            float2 nv[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) nv[r] = make_float2(r == jj ? 1.f : 0.f, 0.f);
#pragma unroll
            for (int r = 1; r < 16; ++r) {
                float2 s = make_float2(0.f, 0.f);
#pragma unroll
                for (int s2 = 0; s2 < r; ++s2) {
                    const float2 l = sm.g2[(p * 16 + r) * LDG + p * 16 + s2];
                    s.x += l.x * nv[s2].x - l.y * nv[s2].y;
                    s.y += l.x * nv[s2].y + l.y * nv[s2].x;
                }
                const float bt = sm.beta[p * 16 + r];
                if (r > jj) nv[r] = make_float2(-bt * s.x, -bt * s.y);
            }
            if (lane < 16) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (r > jj) sm.g2[(p * 16 + r) * LDG + p * 16 + jj] = nv[r];
            }
        }
        __syncthreads();
        // off-diagonal blocks, block row by block row:
        //   N_ps = -N_pp sum_{qb = s}^{p-1} (D_beta L')_{p qb} N_{qb s}
#pragma unroll
        for (int p = 1; p < NRB; ++p) {
            f32x4 res[2];
            const int ntask = 2 * p;
#pragma unroll
            for (int it = 0; it < 2; ++it) {
                const int task = wave + 4 * it;
                if (task < ntask) {
                    const int s = task >> 1, h = task & 1;
                    const int row = p * 16 + c;
                    const float brow = sm.beta[row];
                    const int jcol = s * 16 + h * 8 + (c >> 1);
                    f32x4 acc = zero4();
                    for (int qb = s; qb < p; ++qb) {
                        Frag8 a, b;
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int kk = qb * 16 + 4 * g + r;
                            const float2 l = sm.g2[row * LDG + kk];
                            a.v[2 * r] = brow * l.x;
                            a.v[2 * r + 1] = brow * l.y;
                            float2 y = sm.g2[kk * LDG + jcol];
                            if (qb == s) y = kk > jcol ? y : make_float2(kk == jcol ? 1.f : 0.f, 0.f);
                            bpair(b, r, y.x, y.y, qp);
                        }
                        mma<PREC_F32>(acc, a, b);
                    }
                    const Frag8 bx = bfrag_from_acc(acc, qp);
                    Frag8 a;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int kk = 4 * g + r;
                        float2 l = sm.g2[row * LDG + p * 16 + kk];
                        l = kk < c ? l : make_float2(kk == c ? 1.f : 0.f, 0.f);
                        a.v[2 * r] = l.x;
                        a.v[2 * r + 1] = l.y;
                    }
                    f32x4 acc2 = zero4();
                    mma<PREC_F32>(acc2, a, bx);
                    res[it] = -acc2;
                }
            }
            __syncthreads();
#pragma unroll
            for (int it = 0; it < 2; ++it) {
                const int task = wave + 4 * it;
                if (task < ntask) {
                    const int s = task >> 1, h = task & 1;
                    const int jcol = s * 16 + h * 8 + (c >> 1);
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        g2f[2 * ((p * 16 + 4 * g + r) * LDG + jcol) + qp] = res[it][r];
                }
            }
            __syncthreads();
        }

        // ============================================================ W: U and Wt
        // A fragment of T = N D_beta: rows rb*16 + c, K-block kb
        auto tfrag = [&](int rb, int kb) {
            Frag8 a;
            const int row = rb * 16 + c;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int j = kb * 16 + 4 * g + r;
                float2 nvv = sm.g2[row * LDG + j];
                nvv = j < row ? nvv : make_float2(j == row ? 1.f : 0.f, 0.f);
                const float bj = sm.beta[j];
                a.v[2 * r] = nvv.x * bj;
                a.v[2 * r + 1] = nvv.y * bj;
            }
            return a;
        };
        f32x4 D[CBW][NRB];
        {
            Frag8 bv[CBW][NRB];
#pragma unroll
            for (int w = 0; w < CBW; ++w)
#pragma unroll
                for (int kb = 0; kb < NRB; ++kb)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        bpair(bv[w][kb], r, vf[w][kb][r].x, -vf[w][kb][r].y, qp);   // conj(v)
#pragma unroll
            for (int w = 0; w < CBW; ++w)
#pragma unroll
                for (int rb = 0; rb < NRB; ++rb) D[w][rb] = zero4();
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
                for (int kb = 0; kb <= rb; ++kb) {
                    const Frag8 a = tfrag(rb, kb);
#pragma unroll
                    for (int w = 0; w < CBW; ++w)
                        if (wave + 4 * w < ncb) mma<P>(D[w][rb], a, bv[w][kb]);
                }
        }
        {
            constexpr int NWT = NRB * (2 * MP / 16);         // Wt tiles
            constexpr int PER = (NWT + 3) / 4;
            f32x4 wres[PER];
#pragma unroll
            for (int it = 0; it < PER; ++it) {
                const int tile = wave + 4 * it;
                wres[it] = zero4();
                if (tile < NWT) {
                    const int rb = tile / (2 * MP / 16);
                    const int ib = tile - rb * (2 * MP / 16);
                    const int icol = ib * 8 + (c >> 1);
                    for (int kb = 0; kb <= rb; ++kb) {
                        const Frag8 a = tfrag(rb, kb);
                        Frag8 b;
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const float2 y = sm.kg[(kb * 16 + 4 * g + r) * LDX + icol];
                            bpair(b, r, y.x, y.y, qp);
                        }
                        mma<P>(wres[it], a, b);
                    }
                }
            }
            __syncthreads();
#pragma unroll
            for (int it = 0; it < PER; ++it) {
                const int tile = wave + 4 * it;
                if (tile < NWT) {
                    const int rb = tile / (2 * MP / 16);
                    const int ib = tile - rb * (2 * MP / 16);
                    const int icol = ib * 8 + (c >> 1);
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        kgf[2 * ((rb * 16 + 4 * g + r) * LDX + icol) + qp] = wres[it][r];
                }
            }
            __syncthreads();
        }

        // ============================================================ D: Delta, O, S update
#pragma unroll
        for (int w = 0; w < CBW; ++w) {
            const int cb = wave + 4 * w;
            if (cb >= ncb) continue;
            const int jl = cb * 8 + (c >> 1);
            const int j = n0 + jl;
            Frag8 sb[MP / 16];
#pragma unroll
            for (int kb = 0; kb < MP / 16; ++kb) sb[kb] = bfrag_from_acc(Sacc[w][kb], qp);
            // Delta = U - Wt S
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb) {
                f32x4 pw = zero4();
#pragma unroll
                for (int kb = 0; kb < MP / 16; ++kb) {
                    Frag8 a;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float2 x = sm.kg[(rb * 16 + c) * LDX + kb * 16 + 4 * g + r];
                        a.v[2 * r] = x.x;
                        a.v[2 * r + 1] = x.y;
                    }
                    mma<P>(pw, a, sb[kb]);
                }
                D[w][rb] = D[w][rb] - pw;
            }
            Frag8 db[NRB];
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb) db[rb] = bfrag_from_acc(D[w][rb], qp);
            // O^* = conj(Q)G S + tril(A) Delta ; o = conj(O^*)
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb) {
                f32x4 acc = zero4();
                const int row = rb * 16 + c;
#pragma unroll
                for (int kb = 0; kb < MP / 16; ++kb) {
                    Frag8 a;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float2 x = sm.qg[row * LDX + kb * 16 + 4 * g + r];
                        a.v[2 * r] = x.x;
                        a.v[2 * r + 1] = x.y;
                    }
                    mma<P>(acc, a, sb[kb]);
                }
#pragma unroll
                for (int jb = 0; jb <= rb; ++jb) {
                    Frag8 a;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int jt = jb * 16 + 4 * g + r;
                        const float2 lo = sm.g2[jt * LDG + row];      // A[row][jt] stored transposed
                        const float2 dg = sm.g2[row * LDG + row];     // A diagonal
                        const float2 lo_p = pin(lo), dg_p = pin(dg);
                        const float2 x = masked(jt <= row, jt < row ? lo_p : dg_p);
                        a.v[2 * r] = x.x;
                        a.v[2 * r + 1] = x.y;
                    }
                    mma<P>(acc, a, db[jb]);
                }
                if (j < n && go != nullptr) {     // o == NULL: no output
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int t = t0 + rb * 16 + 4 * g + r;
                        if (t < T)
                            Elem<TOUT>::store(go, 2 * (base_tn + static_cast<long>(t) * n + j) + qp,
                                              qp ? -acc[r] : acc[r]);
                    }
                }
            }
            // S = diag(g_C) S + diag(g_C) (K/G)^T Delta
#pragma unroll
            for (int kb = 0; kb < MP / 16; ++kb) {
                const int irow = kb * 16 + c;
                const float2 gcr = sm.gc[irow];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float2 gg = sm.gc[kb * 16 + 4 * g + r];
                    const float own = Sacc[w][kb][r];
                    const float oth = partner(own);
                    Sacc[w][kb][r] = qp ? (gg.x * own + gg.y * oth) : (gg.x * own - gg.y * oth);
                }
#pragma unroll
                for (int tb = 0; tb < NRB; ++tb) {
                    Frag8 a;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float2 x = sm.ki[(tb * 16 + 4 * g + r) * LDX + irow];
                        a.v[2 * r] = x.x * gcr.x - x.y * gcr.y;
                        a.v[2 * r + 1] = x.x * gcr.y + x.y * gcr.x;
                    }
                    mma<P>(Sacc[w][kb], a, db[tb]);
                }
            }
        }
        __syncthreads();
    }

    // ---------------------------------------------------------------- final state
    if (args.S_T != nullptr) {
#pragma unroll
        for (int w = 0; w < CBW; ++w) {
            const int cb = wave + 4 * w;
            const int j = n0 + cb * 8 + (c >> 1);
            if (cb >= ncb || j >= n) continue;
#pragma unroll
            for (int kb = 0; kb < MP / 16; ++kb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = kb * 16 + 4 * g + r;
                    if (i < m) args.S_T[2 * (base_mn + static_cast<long>(i) * n + j) + qp] = Sacc[w][kb][r];
                }
        }
    }
}

template <int P, typename TIN, typename TOUT>
static hipError_t launch_chunk_t(const ChunkLaunch& L, hipStream_t st)
{
    ChunkArgs a;
    a.q = L.q; a.k = L.k; a.v = L.v; a.alpha = L.alpha; a.theta = L.theta; a.beta = L.beta;
    a.S0 = L.S0; a.o = L.o; a.S_T = L.S_T;
    a.T = L.T; a.m = L.m; a.n = L.n; a.slice = L.slice;
    a.n_slices = (L.n + L.slice - 1) / L.slice;
    a.amin = L.alpha_min; a.aspan = L.alpha_max - L.alpha_min; a.tmax = L.theta_max; a.eps = L.eps;
    const dim3 grid(static_cast<unsigned>(static_cast<long>(L.B) * L.H * a.n_slices));
    auto go = [&](auto gated) {
        constexpr bool G = decltype(gated)::value;
        switch (L.C) {
            case 16: hipLaunchKernelGGL((chunk_kernel<P, TIN, TOUT, 16, G>), grid, dim3(NTHR), 0, st, a); break;
            case 32: hipLaunchKernelGGL((chunk_kernel<P, TIN, TOUT, 32, G>), grid, dim3(NTHR), 0, st, a); break;
            case 64: hipLaunchKernelGGL((chunk_kernel<P, TIN, TOUT, 64, G>), grid, dim3(NTHR), 0, st, a); break;
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    };
    return L.gated ? go(std::true_type{}) : go(std::false_type{});
}

hipError_t launch_chunk(const ChunkLaunch& L, hipStream_t st)
{
    if (L.in_bf16) return launch_chunk_bf16(L, st);
    return L.out_bf16 ? launch_chunk_t<PREC_F32, float, uint16_t>(L, st)
                      : launch_chunk_t<PREC_F32, float, float>(L, st);
}

}  // namespace sfda
