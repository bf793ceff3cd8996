// Chunkwise SFDA forward for bfloat16 inputs on gfx950: a producer/consumer pipeline inside
// one workgroup per (batch, head, slice of value columns).
//
// Method.  Inside a chunk of C tokens, with g_t = lambda_1 ... lambda_t (the diagonal of
// Gamma_t) and S the state entering the chunk, the recurrence reads
// S_t = Lambda_t S_{t-1} + k_t delta_t with delta_t = beta_t (v_t^* - k_t^* Lambda_t S_{t-1}).
// Unrolling it gives the chunk-WY factors of Thm 4.2 / Cor. 4.3 in closed form and
//   (I + D_beta L') Delta = D_beta (conj(V) - (conj(K) * G) S)             (i)
//   L'[t, j] = k_t^* diag(g_t / g_j) k_j  (j < t)
//   O^*   = (conj(Q) * G) S + tril(A) Delta,  A[r, j] = q_r^* diag(g_r / g_j) k_j  (j <= r)
//   S_out = diag(g_C) (S + (K / G)^T Delta)
// i.e. the exact affine chunk transfer of Thm 4.4 (the paper's M is (I + L' D_beta)^{-1})
// with the prefix outputs of Thm 4.5, applied by the boundary-state scan (apply-transfer
// equation, Thm 6.1).  Equation (i) is solved per chunk by blocked forward substitution:
// with 16 x 16 blocks, Delta_p = N_pp (R_p - sum_{q<p} (D_beta L')_pq Delta_q) where
// N_pp = (I + (D_beta L')_pp)^{-1}.  The state-independent work is therefore the cumulative
// phase-decay g, the operands conj(Q)G, conj(K)G, K/G, the Gram blocks of L' and A, and the
// four 16 x 16 inverses N_pp; the state-dependent work is five small complex GEMMs.
//
// Pipeline (512 threads = 8 waves, two per SIMD):
//   waves 0-3 (consumers) own value columns and hold their columns of S in MFMA
//     accumulators for the whole scan; for chunk c they compute Delta, O and S_out;
//   waves 4-7 (producers) prepare chunk c + 1: phase 1 loads q, k, alpha, theta, beta
//     (prefetched a chunk ahead), forms g from running sums of log alpha and theta and
//     writes conj(Q)G, conj(K)G, K/G (bf16) to LDS; phase 2 forms the Gram blocks of L' and
//     A on MFMA (wave p owns token block p) and inverts its diagonal block of D_beta L'.
//   Operands live in two LDS sets (chunk c and chunk c + 1); two barriers per chunk.
//
// LDS layouts.  A C x 64 complex bf16 array has rows padded from 256 to 272 bytes; a
// 16 x 16 complex bf16 block has 64-byte rows whose 16-byte chunks are XOR-swizzled by
// (row >> 2) & 3.  Either way one MFMA operand fragment (4 consecutive complex values of one
// row) is a single conflict-free 16-byte read.
//
// Complex products use the real-block form of sfda_device.h on v_mfma_f32_16x16x32_bf16
// with fp32 accumulation; the diagonal inverses are computed in fp32.
#include "sfda_device.h"
#include "sfda_launch.h"

namespace sfda {
namespace pipe {

constexpr int MP = 64;          // key channels per workgroup (m zero-padded)
constexpr int NTH = 512;

typedef uint32_t u32;
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ bf16x8 as_bf(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }
__device__ __forceinline__ u32 pack_bf16(float lo, float hi) {
    bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(u32, v);
}
__device__ __forceinline__ float bf_lo(u32 w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(u32 w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ u32 pin_u(u32 x) { asm volatile("" : "+v"(x)); return x; }

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(a), as_bf(b), c, 0, 0, 0);
}

// B fragment (Ybig entries) from four complex bf16 values y[r] = Y(4g + r, j):
// q = 0: (Re, -Im); q = 1: (Im, Re).
// qmask = 0xFFFFFFFF when q = 1, else 0 (lane parity, computed once per lane).
__device__ __forceinline__ u32x4 ybig(u32x4 y, u32 qmask) {
    u32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const u32 sw = __builtin_amdgcn_alignbit(y[k], y[k], 16);   // (Im, Re)
        const u32 ng = y[k] ^ 0x80000000u;                          // (Re, -Im)
        r[k] = ng ^ ((sw ^ ng) & qmask);
    }
    return r;
}

// B fragment from an accumulator tile whose rows are the next product's K-block.
// nsign = 0x80000000 when q = 0 (the partner's imaginary part enters negated), else 0.
__device__ __forceinline__ u32x4 bfrag(const f32x4& acc, u32 nsign) {
    u32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float own = acc[k];
        const float oth = __uint_as_float(__float_as_uint(partner(own)) ^ nsign);
        r[k] = pack_bf16(own, oth);
    }
    return r;
}
__device__ __forceinline__ float flip(float x, u32 sign) { return __uint_as_float(__float_as_uint(x) ^ sign); }

// ------------------------------------------------------------------ LDS addressing (bytes)

// C x 64 complex bf16, row-major, rows padded to 272 bytes (68 words: consecutive rows start
// 4 banks apart, so 16 rows x one 16-byte chunk, or 16 consecutive words of 4 rows spaced
// 4 apart, touch 64 distinct banks).  Offsets are linear in row and column, so every
// fragment address is one lane base plus an immediate.
constexpr int RP = 272;
__device__ __forceinline__ int rm_off(int row, int i) { return row * RP + i * 4; }
__device__ __forceinline__ int rm_frag(int row, int chunk) { return row * RP + chunk * 16; }
// 16 x 16 complex bf16 block
__device__ __forceinline__ int blk_off(int row, int j) {
    return row * 64 + ((((j >> 2) ^ (row >> 2)) & 3) << 4) + ((j & 3) << 2);
}
__device__ __forceinline__ int blk_frag(int row, int chunk) {
    return row * 64 + (((chunk ^ (row >> 2)) & 3) << 4);
}

template <int C>
struct Smem {
    static constexpr int NRB = C / 16;
    static constexpr int NLB = NRB * (NRB - 1) / 2 > 0 ? NRB * (NRB - 1) / 2 : 1;
    static constexpr int NAQ = NRB * (NRB + 1) / 2;
    struct Set {
        u32x4 qg[C * RP / 16];   // conj(q) g      [t][i]
        u32x4 kg[C * RP / 16];   // conj(k) g      [t][i]
        u32x4 ki[C * RP / 16];   // k / g          [t][i]
        u32x4 lb[NLB * 64];      // -(D_beta L') off-diagonal blocks (p > q)
        u32x4 nd[NRB * 64];      // N_pp = (I + (D_beta L')_pp)^{-1}
        u32x4 aq[NAQ * 64];      // A lower blocks, zero above the diagonal
        float beta[C];
        float2 gc[MP];           // g_C
    };
    Set set[2];
    float scr[4][16 * 16 * 2];   // per producer wave: diagonal block of L' (fp32)
};

struct Args {
    const uint16_t *q, *k, *v, *alpha, *theta, *beta;
    const float* S0;
    void* o;
    float* S_T;
    int T, m, n, n_slices, slice;
};

template <typename TOUT, int C>
__global__ __launch_bounds__(NTH, 1) void chunk_pipe_kernel(Args args)
{
    constexpr int NRB = C / 16;
    constexpr int SEGT = C / 4;          // tokens per producer lane
    __shared__ Smem<C> sm;
    char* const smb = reinterpret_cast<char*>(&sm);

    const int T = args.T, m = args.m, n = args.n;
    const long bh = blockIdx.x / args.n_slices;
    const int sl = blockIdx.x - static_cast<int>(bh) * args.n_slices;
    const int n0 = sl * args.slice;
    const int ncb = (min(args.slice, n - n0) + 7) / 8;     // active 8-column blocks
    const int nchunks = (T + C - 1) / C;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int c = lane & 15;
    const int g = lane >> 4;
    const int qp = lane & 1;
    const u32 qmask = qp ? 0xFFFFFFFFu : 0u;
    const u32 nsign = qp ? 0u : 0x80000000u;      // negates where q = 0
    const u32 csign = qp ? 0x80000000u : 0u;      // negates where q = 1 (conjugation)
    const bool consumer = wave < 4;

    const long base_tm = bh * static_cast<long>(T) * m;
    const long base_tn = bh * static_cast<long>(T) * n;
    const long base_mn = bh * static_cast<long>(m) * n;
    const long base_t = bh * static_cast<long>(T);

    auto set_off = [&](int s) -> char* { return reinterpret_cast<char*>(&sm.set[s]); };

    // ---------------------------------------------------------------- consumer state
    f32x4 Sacc[2][4];        // columns cb = wave + 4 w, rows kb*16 + 4g + r
    u32x4 db[2][NRB];        // Delta as B fragments
    u32 vv[2][NRB][2];       // prefetched v: this lane's part of 4 tokens, two bf16 per word
    // ---------------------------------------------------------------- producer state
    u32 pa[SEGT / 2], pt[SEGT / 2];   // alpha, theta bits, two tokens per word
    u32 pq[SEGT], pk[SEGT];           // q, k (one complex bf16 per word)
    u32 pbeta = 0;

    const int cbw0 = wave, cbw1 = wave + 4;   // consumer column blocks
    auto cb_active = [&](int w) { return (w == 0 ? cbw0 : cbw1) < ncb; };

    auto load_v = [&](int ch) {
        const int t0 = ch * C;
#pragma unroll
        for (int w = 0; w < 2; ++w) {
            const int cb = w == 0 ? cbw0 : cbw1;
            const int j = n0 + cb * 8 + (c >> 1);
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
                for (int r2 = 0; r2 < 2; ++r2) {
                    u32 word = 0;
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int t = t0 + rb * 16 + 4 * g + 2 * r2 + h;
                        const bool ok = cb < ncb && j < n && t < T;
                        const long e = 2 * (base_tn + static_cast<long>(min(t, T - 1)) * n + min(j, n - 1)) + qp;
                        const u32 x = pin_u(args.v[e]);
                        word |= (ok ? x : 0u) << (16 * h);
                    }
                    vv[w][rb][r2] = word;
                }
        }
    };

    const int pw = wave - 4;                   // producer wave index
    const int pch = (pw & 3) * 16 + c;         // producer channel
    const int psg = g;                         // producer token segment

    auto load_p = [&](int ch) {
        const int t0 = ch * C;
        const int i = min(pch, m - 1);
#pragma unroll
        for (int u = 0; u < SEGT; ++u) {
            const int t = min(t0 + psg * SEGT + u, T - 1);
            const long e = base_tm + static_cast<long>(t) * m + i;
            const u32 av = args.alpha[e], tv = args.theta[e];
            if (u & 1) {
                pa[u >> 1] |= av << 16;
                pt[u >> 1] |= tv << 16;
            } else {
                pa[u >> 1] = av;
                pt[u >> 1] = tv;
            }
            pq[u] = *reinterpret_cast<const u32*>(args.q + 2 * e);
            pk[u] = *reinterpret_cast<const u32*>(args.k + 2 * e);
        }
        pbeta = args.beta[base_t + min(t0 + (lane & (C - 1)), T - 1)];
    };

    // ---------------------------------------------------------------- producer phases
    auto produce1 = [&](int ch) {          // operands of chunk ch into set ch & 1
        char* S = set_off(ch & 1);
        auto& st = sm.set[ch & 1];
        const int t0 = ch * C;
        const bool chan_ok = pch < m;
        auto alpha_at = [&](int u) {
            const bool ok = chan_ok && (t0 + psg * SEGT + u) < T;
            const u32 w = pa[u >> 1];
            return ok ? ((u & 1) ? bf_hi(w) : bf_lo(w)) : 1.f;
        };
        auto theta_at = [&](int u) {
            const bool ok = chan_ok && (t0 + psg * SEGT + u) < T;
            const u32 w = pt[u >> 1];
            return ok ? ((u & 1) ? bf_hi(w) : bf_lo(w)) : 0.f;
        };
        float sa = 0.f, sp = 0.f;      // segment totals (first pass)
#pragma unroll
        for (int u = 0; u < SEGT; ++u) {
            sa += __logf(alpha_at(u));
            sp += theta_at(u);
        }
        // exclusive prefix over the four token segments of this channel (lane groups)
        float pre_a = 0.f, pre_p = 0.f;
#pragma unroll
        for (int d = 1; d < 4; ++d) {
            const int src = ((psg - d) & 3) * 16 + c;
            const float ya = __shfl(sa, src);
            const float yp = __shfl(sp, src);
            if (psg >= d) { pre_a += ya; pre_p += yp; }
        }
        float A = pre_a, Ph = pre_p;   // running sums (second pass, same order as the first)
#pragma unroll
        for (int u = 0; u < SEGT; ++u) {
            const int tl = psg * SEGT + u;
            const bool ok = chan_ok && (t0 + tl) < T;
            A += __logf(alpha_at(u));
            Ph += theta_at(u);
            const float e = __expf(A), ei = __expf(-A);
            float sn, cs;
            __sincosf(Ph, &sn, &cs);
            const float gr = e * cs, gi = e * sn;
            const float hr = ei * cs, hi = -ei * sn;
            const u32 qw = ok ? pq[u] : 0u, kw = ok ? pk[u] : 0u;
            const float qr = bf_lo(qw), qi = bf_hi(qw), kr = bf_lo(kw), ki = bf_hi(kw);
            *reinterpret_cast<u32*>(S + offsetof(typename Smem<C>::Set, qg) + rm_off(tl, pch)) =
                pack_bf16(qr * gr + qi * gi, qr * gi - qi * gr);
            *reinterpret_cast<u32*>(S + offsetof(typename Smem<C>::Set, kg) + rm_off(tl, pch)) =
                pack_bf16(kr * gr + ki * gi, kr * gi - ki * gr);
            *reinterpret_cast<u32*>(S + offsetof(typename Smem<C>::Set, ki) + rm_off(tl, pch)) =
                pack_bf16(kr * hr - ki * hi, kr * hi + ki * hr);
            if (tl == C - 1) st.gc[pch] = make_float2(gr, gi);
        }
        if (pw == 0 && lane < C) st.beta[lane] = (t0 + lane < T) ? bf16_bits_to_f32(static_cast<uint16_t>(pbeta)) : 0.f;
    };

    auto produce2_blocks = [&](int ch) {   // Gram blocks and diagonal inverses of chunk ch
        if (pw >= NRB) return;
        char* S = set_off(ch & 1);
        auto& st = sm.set[ch & 1];
        const int rb = pw;
        u32x4 akg[4], aqg[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            akg[kb] = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, kg) + rm_frag(rb * 16 + c, kb * 4 + g));
            aqg[kb] = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, qg) + rm_frag(rb * 16 + c, kb * 4 + g));
        }
        float* scr = sm.scr[pw];
        for (int jb = 0; jb <= rb; ++jb) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int jl = h * 8 + (c >> 1);          // column inside block jb
                const int j = jb * 16 + jl;
                f32x4 accL = zero4(), accA = zero4();
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const u32x4 y = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, ki) + rm_frag(j, kb * 4 + g));
                    const u32x4 bk = ybig(y, qmask);
                    accL = mfma(akg[kb], bk, accL);
                    accA = mfma(aqg[kb], bk, accA);
                }
                char* aqb = S + offsetof(typename Smem<C>::Set, aq) + (rb * (rb + 1) / 2 + jb) * 1024;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int tl = 4 * g + r;
                    const float va = (jb < rb || jl <= tl) ? accA[r] : 0.f;
                    *reinterpret_cast<__bf16*>(aqb + blk_off(tl, jl) + 2 * qp) = static_cast<__bf16>(va);
                    if (jb < rb) {
                        const float bt = st.beta[rb * 16 + tl];
                        char* lbb = S + offsetof(typename Smem<C>::Set, lb) + (rb * (rb - 1) / 2 + jb) * 1024;
                        *reinterpret_cast<__bf16*>(lbb + blk_off(tl, jl) + 2 * qp) = static_cast<__bf16>(-bt * accL[r]);
                    } else {
                        scr[(tl * 16 + jl) * 2 + qp] = accL[r];
                    }
                }
            }
        }
        // this wave's writes of its diagonal block must land before its lanes read them
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // N_pp = (I + D_beta L'_pp)^{-1}; lane jj owns column jj (right-looking updates)
        const int jj = lane & 15;
        float2 nv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) nv[r] = make_float2(r == jj ? 1.f : 0.f, 0.f);
#pragma unroll
        for (int s = 0; s < 15; ++s) {
#pragma unroll
            for (int r = s + 1; r < 16; ++r) {
                const float2 l = *reinterpret_cast<const float2*>(&scr[(r * 16 + s) * 2]);
                const float bt = st.beta[rb * 16 + r];
                const float cr = -bt * l.x, ci = -bt * l.y;
                nv[r].x += cr * nv[s].x - ci * nv[s].y;
                nv[r].y += cr * nv[s].y + ci * nv[s].x;
            }
        }
        if (lane < 16) {
            char* ndb = S + offsetof(typename Smem<C>::Set, nd) + rb * 1024;
#pragma unroll
            for (int r = 0; r < 16; ++r)
                *reinterpret_cast<u32*>(ndb + blk_off(r, jj)) = pack_bf16(nv[r].x, nv[r].y);
        }
    };

    auto produce2 = [&](int ch) {
        produce2_blocks(ch);
        // inputs of the next chunk are fetched after this phase's register peak; their
        // latency overlaps the wait at the barrier
        if (ch + 1 < nchunks) load_p(ch + 1);
    };

    // ---------------------------------------------------------------- consumer phases
    auto consume1 = [&](int ch) {          // Delta of chunk ch
        const char* S = set_off(ch & 1);
        const auto& st = sm.set[ch & 1];
        u32x4 sb[2][4];          // S as B fragments
#pragma unroll
        for (int w = 0; w < 2; ++w)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) sb[w][kb] = bfrag(Sacc[w][kb], nsign);
        // block by block: R_p = beta (conj(V) - Kg S)_p, then
        // Delta_p = N_pp (R_p + sum_{q<p} (-(D_beta L'))_pq Delta_q)
#pragma unroll
        for (int p = 0; p < NRB; ++p) {
            f32x4 acc[2] = {zero4(), zero4()};
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, kg) + rm_frag(p * 16 + c, kb * 4 + g));
                if (cb_active(0)) acc[0] = mfma(a, sb[0][kb], acc[0]);
                if (cb_active(1)) acc[1] = mfma(a, sb[1][kb], acc[1]);
            }
            const float4 bt = *reinterpret_cast<const float4*>(&st.beta[p * 16 + 4 * g]);
            const float btr[4] = {bt.x, bt.y, bt.z, bt.w};
#pragma unroll
            for (int w = 0; w < 2; ++w)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const u32 word = vv[w][p][r >> 1];
                    const float vx = flip((r & 1) ? bf_hi(word) : bf_lo(word), csign);
                    acc[w][r] = btr[r] * (vx - acc[w][r]);
                }
#pragma unroll
            for (int q2 = 0; q2 < p; ++q2) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, lb) + (p * (p - 1) / 2 + q2) * 1024 + blk_frag(c, g));
                if (cb_active(0)) acc[0] = mfma(a, db[0][q2], acc[0]);
                if (cb_active(1)) acc[1] = mfma(a, db[1][q2], acc[1]);
            }
            const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, nd) + p * 1024 + blk_frag(c, g));
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                f32x4 d = zero4();
                if (cb_active(w)) d = mfma(a, bfrag(acc[w], nsign), d);
                db[w][p] = bfrag(d, nsign);
            }
        }
    };

    TOUT* const go = static_cast<TOUT*>(args.o);
    auto consume2 = [&](int ch) {          // outputs and state update of chunk ch
        const char* S = set_off(ch & 1);
        const auto& st = sm.set[ch & 1];
        const int t0 = ch * C;
        u32x4 sb[2][4];          // S (still the chunk-start state) as B fragments
#pragma unroll
        for (int w = 0; w < 2; ++w)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) sb[w][kb] = bfrag(Sacc[w][kb], nsign);
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            f32x4 acc[2] = {zero4(), zero4()};
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, qg) + rm_frag(rb * 16 + c, kb * 4 + g));
                if (cb_active(0)) acc[0] = mfma(a, sb[0][kb], acc[0]);
                if (cb_active(1)) acc[1] = mfma(a, sb[1][kb], acc[1]);
            }
#pragma unroll
            for (int jb = 0; jb <= rb; ++jb) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, aq) + (rb * (rb + 1) / 2 + jb) * 1024 + blk_frag(c, g));
                if (cb_active(0)) acc[0] = mfma(a, db[0][jb], acc[0]);
                if (cb_active(1)) acc[1] = mfma(a, db[1][jb], acc[1]);
            }
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                const int cb = w == 0 ? cbw0 : cbw1;
                const int j = n0 + cb * 8 + (c >> 1);
                if (cb < ncb && j < n) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int t = t0 + rb * 16 + 4 * g + r;
                        if (t < T)
                            Elem<TOUT>::store(go, 2 * (base_tn + static_cast<long>(t) * n + j) + qp,
                                              flip(acc[w][r], csign));
                    }
                }
            }
        }
        // S <- diag(g_C) (S + (K/G)^T Delta)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            const int irow = kb * 16 + c;
#pragma unroll
            for (int tb = 0; tb < NRB; ++tb) {
                u32x4 a;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    a[r] = *reinterpret_cast<const u32*>(S + offsetof(typename Smem<C>::Set, ki) + rm_off(tb * 16 + 4 * g + r, irow));
                if (cb_active(0)) Sacc[0][kb] = mfma(a, db[0][tb], Sacc[0][kb]);
                if (cb_active(1)) Sacc[1][kb] = mfma(a, db[1][tb], Sacc[1][kb]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float2 gg = st.gc[kb * 16 + 4 * g + r];
#pragma unroll
                for (int w = 0; w < 2; ++w) {
                    const float own = Sacc[w][kb][r];
                    const float oth = partner(own);
                    Sacc[w][kb][r] = gg.x * own + flip(gg.y, nsign) * oth;
                }
            }
        }
        if (ch + 1 < nchunks) load_v(ch + 1);
    };

    // ---------------------------------------------------------------- roles
    // The role test is wave-uniform and encloses each role's whole life (prologue, chunk
    // loop, epilogue), so each role keeps only its own registers live.  Both loops pass the
    // same sequence of workgroup barriers: two per chunk plus the producers' lead-in chunk.
    if (consumer) {
#pragma unroll
        for (int w = 0; w < 2; ++w) {
            const int cb = w == 0 ? cbw0 : cbw1;
            const int j = n0 + cb * 8 + (c >> 1);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = kb * 16 + 4 * g + r;
                    float x = 0.f;
                    if (args.S0 != nullptr)
                        x = masked(cb < ncb && j < n && i < m,
                                   args.S0[2 * (base_mn + static_cast<long>(min(i, m - 1)) * n + min(j, n - 1)) + qp]);
                    Sacc[w][kb][r] = x;
                }
        }
        if (nchunks > 0) load_v(0);
        for (int ch = -1; ch < nchunks; ++ch) {
            if (ch >= 0) consume1(ch);
            __syncthreads();
            if (ch >= 0) consume2(ch);
            __syncthreads();
        }
        if (args.S_T != nullptr) {
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                const int cb = w == 0 ? cbw0 : cbw1;
                const int j = n0 + cb * 8 + (c >> 1);
                if (cb >= ncb || j >= n) continue;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int i = kb * 16 + 4 * g + r;
                        if (i < m) args.S_T[2 * (base_mn + static_cast<long>(i) * n + j) + qp] = Sacc[w][kb][r];
                    }
            }
        }
    } else {
        if (nchunks > 0) load_p(0);
        for (int ch = -1; ch < nchunks; ++ch) {
            if (ch + 1 < nchunks) produce1(ch + 1);
            __syncthreads();
            if (ch + 1 < nchunks) produce2(ch + 1);
            __syncthreads();
        }
    }
}

template <typename TOUT>
static hipError_t launch_t(const ChunkLaunch& L, hipStream_t st)
{
    Args a;
    a.q = static_cast<const uint16_t*>(L.q);
    a.k = static_cast<const uint16_t*>(L.k);
    a.v = static_cast<const uint16_t*>(L.v);
    a.alpha = static_cast<const uint16_t*>(L.alpha);
    a.theta = static_cast<const uint16_t*>(L.theta);
    a.beta = static_cast<const uint16_t*>(L.beta);
    a.S0 = L.S0; a.o = L.o; a.S_T = L.S_T;
    a.T = L.T; a.m = L.m; a.n = L.n; a.slice = L.slice;
    a.n_slices = (L.n + L.slice - 1) / L.slice;
    const dim3 grid(static_cast<unsigned>(static_cast<long>(L.B) * L.H * a.n_slices));
    switch (L.C) {
        case 16: hipLaunchKernelGGL((chunk_pipe_kernel<TOUT, 16>), grid, dim3(NTH), 0, st, a); break;
        case 32: hipLaunchKernelGGL((chunk_pipe_kernel<TOUT, 32>), grid, dim3(NTH), 0, st, a); break;
        case 64: hipLaunchKernelGGL((chunk_pipe_kernel<TOUT, 64>), grid, dim3(NTH), 0, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace pipe

hipError_t launch_chunk_bf16(const ChunkLaunch& L, hipStream_t st)
{
    return L.out_bf16 ? pipe::launch_t<uint16_t>(L, st) : pipe::launch_t<float>(L, st);
}

}  // namespace sfda
