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
#include <utility>

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
template <typename TOUT> __device__ __forceinline__ TOUT to_out(float x);
template <> __device__ __forceinline__ float to_out<float>(float x) { return x; }
template <> __device__ __forceinline__ uint16_t to_out<uint16_t>(float x) { return f32_to_bf16_bits(x); }
__device__ __forceinline__ float bf_lo(u32 w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(u32 w) { return __uint_as_float(w & 0xFFFF0000u); }

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

// One step of the 16 x 16 unit-lower-triangular inverse (see produce2_blocks): lane (g, jj)
// holds rows 4g .. 4g+3 of column jj of N in nv and rows 4g .. 4g+3 of X = -(D_beta L') in
// the accumulator tiles xd (real column c of half h).  Step S2 adds X(r, S2) N(S2, jj) to
// every row r > S2.
template <int S2>
__device__ __forceinline__ void inverse_step(float2 (&nv)[4], const f32x4 (&xd)[2], int g, int jj)
{
    const int src = ((S2 >> 2) * 16 + jj) * 4;            // lane holding N(S2, jj)
    const float2 own = nv[S2 & 3];
    const float pr = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(own.x)));
    const float pi = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(own.y)));
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        // X(4g + r, S2): Re at lane 2 (S2 & 7), Im at lane 2 (S2 & 7) + 1 of this 16-lane row
        const int xv = __float_as_int(xd[S2 >> 3][r]);
        const float xr = __int_as_float(__builtin_amdgcn_update_dpp(0, xv, 0x150 + 2 * (S2 & 7), 0xF, 0xF, false));
        const float xi = __int_as_float(__builtin_amdgcn_update_dpp(0, xv, 0x151 + 2 * (S2 & 7), 0xF, 0xF, false));
        const bool below = 4 * g + r > S2;
        nv[r].x += below ? xr * pr - xi * pi : 0.f;
        nv[r].y += below ? xr * pi + xi * pr : 0.f;
    }
}
template <int... S>
__device__ __forceinline__ void inverse_steps(float2 (&nv)[4], const f32x4 (&xd)[2], int g, int jj,
                                              std::integer_sequence<int, S...>)
{
    (inverse_step<S>(nv, xd, g, jj), ...);
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
    u32x4 ostage[4][128];        // per consumer wave: one 16-row output tile (<= 2 KiB)
};

struct Args {
    const uint16_t *q, *k, *v, *alpha, *theta, *beta;
    const float* S0;
    void* o;
    float* S_T;
    int T, m, n, n_slices, slice;
};

// CBW: 8-column blocks of S per consumer wave (2 for 64-column slices, 1 for <= 32).
template <typename TOUT, int C, int CBW>
__global__ __launch_bounds__(NTH, 1) void chunk_pipe_kernel(Args args)
{
    constexpr int NRB = C / 16;
    constexpr int TPL = C / 16;          // tokens per producer lane (16 segments of TPL)
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
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar)
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
    f32x4 Sacc[CBW][4];      // columns cb = CBW wave + w, rows kb*16 + 4g + r
    u32x4 db[CBW][NRB];      // Delta as B fragments
    u32 vv[CBW][NRB][2];     // prefetched v: this lane's part of 4 tokens, two bf16 per word
    // ---------------------------------------------------------------- producer state
    // producer lane = 4 channels x TPL tokens; prefetched raw (consumed a phase later)
    uint2 pa[TPL], pt[TPL];           // alpha, theta bits of 4 channels
    u32x4 pq[TPL], pk[TPL];           // q, k of 4 channels (complex bf16)
    u32 pbeta = 0;

    // consumer column block w is cb = CBW wave + w (contiguous); blocks past the slice compute
    // on zeros

    auto load_v = [&](int ch) {
        const int t0 = ch * C;
#pragma unroll
        for (int w = 0; w < CBW; ++w) {
            const int cb = CBW * wave + w;
            const int j = n0 + cb * 8 + (c >> 1);
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
                for (int r2 = 0; r2 < 2; ++r2) {
                    // raw (clamped-index) loads; out-of-range entries are masked where they are
                    // used, one chunk later, so nothing waits on these loads here
                    u32 word = 0;
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int t = t0 + rb * 16 + 4 * g + 2 * r2 + h;
                        const long e = 2 * (base_tn + static_cast<long>(min(t, T - 1)) * n + min(j, n - 1)) + qp;
                        word |= static_cast<u32>(args.v[e]) << (16 * h);
                    }
                    vv[w][rb][r2] = word;
                }
        }
    };

    const int pw = wave - 4;                   // producer wave index
    const int pseg = lane >> 2;                // token segment (tokens pseg*TPL .. +TPL-1)
    const int pc0 = (pw & 3) * 16 + (lane & 3) * 4;   // first of this lane's 4 channels

    auto load_p = [&](int ch) {
        const int t0 = ch * C;
        if ((m & 3) == 0) {     // 4-channel vector loads (8 bytes of alpha/theta, 16 of q/k)
            const int cc = min(pc0, m - 4);
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                const int t = min(t0 + pseg * TPL + u, T - 1);
                const long e = base_tm + static_cast<long>(t) * m + cc;
                pa[u] = *reinterpret_cast<const uint2*>(args.alpha + e);
                pt[u] = *reinterpret_cast<const uint2*>(args.theta + e);
                pq[u] = *reinterpret_cast<const u32x4*>(args.q + 2 * e);
                pk[u] = *reinterpret_cast<const u32x4*>(args.k + 2 * e);
            }
        } else {                // any m: element loads (clamped)
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                const int t = min(t0 + pseg * TPL + u, T - 1);
                const long r0 = base_tm + static_cast<long>(t) * m;
                u32 a4[4], t4[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const long e = r0 + min(pc0 + k, m - 1);
                    a4[k] = args.alpha[e];
                    t4[k] = args.theta[e];
                    pq[u][k] = *reinterpret_cast<const u32*>(args.q + 2 * e);
                    pk[u][k] = *reinterpret_cast<const u32*>(args.k + 2 * e);
                }
                pa[u] = make_uint2(a4[0] | (a4[1] << 16), a4[2] | (a4[3] << 16));
                pt[u] = make_uint2(t4[0] | (t4[1] << 16), t4[2] | (t4[3] << 16));
            }
        }
        pbeta = args.beta[base_t + min(t0 + (lane & (C - 1)), T - 1)];
    };

    // ---------------------------------------------------------------- producer phases
    auto produce1 = [&](int ch) {          // operands of chunk ch into set ch & 1
        char* S = set_off(ch & 1);
        auto& st = sm.set[ch & 1];
        const int t0 = ch * C;
        auto half = [](uint2 w, int k) {       // k-th bf16 of 4 packed in two words
            const u32 x = (k < 2) ? w.x : w.y;
            return (k & 1) ? bf_hi(x) : bf_lo(x);
        };
        // running sums over this lane's TPL tokens, per channel, of log2(alpha) and of theta
        // in revolutions (theta / 2 pi): the hardware exp2 / sin / cos then need no scaling
        constexpr float INV_2PI = 0.15915494309189535f;
        float la[TPL][4], lp[TPL][4];
        float sa[4], sp[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const bool chan_ok = pc0 + k < m;
            float ra = 0.f, rp = 0.f;
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                const bool ok = chan_ok && (t0 + pseg * TPL + u) < T;
                ra += __builtin_amdgcn_logf(ok ? half(pa[u], k) : 1.f);
                rp += ok ? half(pt[u], k) * INV_2PI : 0.f;
                la[u][k] = ra;
                lp[u][k] = rp;
            }
            sa[k] = ra;
            sp[k] = rp;
        }
        // exclusive prefix over the 16 token segments (lanes 4 apart): inclusive scan by
        // doubling, then remove this segment's own total
        float ia[4], ip[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) { ia[k] = sa[k]; ip[k] = sp[k]; }
#pragma unroll
        for (int d = 1; d < 16; d <<= 1) {
            const int src = max(lane - 4 * d, 0);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float ya = __shfl(ia[k], src);
                const float yp = __shfl(ip[k], src);
                if (pseg >= d) { ia[k] += ya; ip[k] += yp; }
            }
        }
#pragma unroll
        for (int u = 0; u < TPL; ++u) {
            const int tl = pseg * TPL + u;
            const bool row_ok = (t0 + tl) < T;
            u32x4 wq, wk, wi;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const bool ok = row_ok && (pc0 + k < m);
                const float A = (ia[k] - sa[k]) + la[u][k];     // log2 of the decay product
                const float Ph = (ip[k] - sp[k]) + lp[u][k];    // phase in revolutions
                const float e = __builtin_amdgcn_exp2f(A), ei = __builtin_amdgcn_exp2f(-A);
                const float sn = __builtin_amdgcn_sinf(Ph), cs = __builtin_amdgcn_cosf(Ph);
                const float gr = e * cs, gi = e * sn;
                const float hr = ei * cs, hi = -ei * sn;
                const u32 qw = ok ? pq[u][k] : 0u, kw = ok ? pk[u][k] : 0u;
                const float qr = bf_lo(qw), qi = bf_hi(qw), kr = bf_lo(kw), ki = bf_hi(kw);
                wq[k] = pack_bf16(qr * gr + qi * gi, qr * gi - qi * gr);
                wk[k] = pack_bf16(kr * gr + ki * gi, kr * gi - ki * gr);
                wi[k] = pack_bf16(kr * hr - ki * hi, kr * hi + ki * hr);
                if (tl == C - 1) st.gc[pc0 + k] = make_float2(gr, gi);
            }
            *reinterpret_cast<u32x4*>(S + offsetof(typename Smem<C>::Set, qg) + rm_off(tl, pc0)) = wq;
            *reinterpret_cast<u32x4*>(S + offsetof(typename Smem<C>::Set, kg) + rm_off(tl, pc0)) = wk;
            *reinterpret_cast<u32x4*>(S + offsetof(typename Smem<C>::Set, ki) + rm_off(tl, pc0)) = wi;
        }
        if (pw == 0 && lane < C) st.beta[lane] = (t0 + lane < T) ? bf16_bits_to_f32(static_cast<uint16_t>(pbeta)) : 0.f;
    };

    // Gram work is split into units (rb, jb), jb <= rb: the 16 x 16 blocks at token block rb,
    // key block jb.  unit_list gives a wave its units: first its own diagonal unit (rb = jb =
    // wave, whose L' block the producer inverts), then an even share of the rest.
    auto unit_list = [&](int wv, int (&units)[3][2]) -> int {
        if (NRB == 4) {
            const int tab[4][3][2] = {{{0, 0}, {3, 0}, {3, 1}}, {{1, 1}, {1, 0}, {3, 2}},
                                      {{2, 2}, {2, 0}, {-1, -1}}, {{3, 3}, {2, 1}, {-1, -1}}};
#pragma unroll
            for (int k = 0; k < 3; ++k) { units[k][0] = tab[wv][k][0]; units[k][1] = tab[wv][k][1]; }
            return wv < 2 ? 3 : 2;
        } else if (NRB == 2) {
            const int tab[4][2] = {{0, 0}, {1, 1}, {1, 0}, {-1, -1}};
            units[0][0] = tab[wv][0]; units[0][1] = tab[wv][1];
            return wv < 3 ? 1 : 0;
        }
        units[0][0] = 0; units[0][1] = 0;
        return wv == 0 ? 1 : 0;
    };
    // one Gram unit: acc[h] (real column block h of key block jb) = X rows rb * (K/G)^T
    auto gram_unit = [&](const char* S, int xoff, int rb, int jb, f32x4 (&acc)[2]) {
        acc[0] = zero4();
        acc[1] = zero4();
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            const u32x4 ax = *reinterpret_cast<const u32x4*>(S + xoff + rm_frag(rb * 16 + c, kb * 4 + g));
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int j = jb * 16 + h * 8 + (c >> 1);
                const u32x4 y = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, ki) + rm_frag(j, kb * 4 + g));
                acc[h] = mfma(ax, ybig(y, qmask), acc[h]);
            }
        }
    };

    auto produce2_blocks = [&](int ch) {   // L' blocks and diagonal inverses of chunk ch
        char* S = set_off(ch & 1);
        auto& st = sm.set[ch & 1];
        f32x4 xd[2];   // -(D_beta L') on the diagonal block (rows 4g + r, real column c of half h)
        int units[3][2];
        const int nu = unit_list(pw, units);
        for (int u = 0; u < nu; ++u) {
            const int rb = units[u][0], jb = units[u][1];
            f32x4 accL[2];
            gram_unit(S, offsetof(typename Smem<C>::Set, kg), rb, jb, accL);
            char* lbb = S + offsetof(typename Smem<C>::Set, lb) + (rb > 0 ? (rb * (rb - 1) / 2 + jb) * 1024 : 0);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int jl = h * 8 + (c >> 1);          // column inside block jb
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int tl = 4 * g + r;
                    const float xb = -st.beta[rb * 16 + tl] * accL[h][r];   // -(D_beta L')
                    if (jb < rb)
                        *reinterpret_cast<__bf16*>(lbb + blk_off(tl, jl) + 2 * qp) = static_cast<__bf16>(xb);
                    else
                        xd[h][r] = xb;                     // diagonal block, kept for the inverse
                }
            }
        }
        if (pw >= NRB) return;
        const int rb = pw;
        // N_pp = (I + D_beta L'_pp)^{-1} by right-looking substitution on all 64 lanes: lane
        // (g, jj) owns rows 4g .. 4g+3 of column jj -- the accumulator layout of xd -- so the
        // entries X(r, s) = -(D_beta L')_rs it needs sit in its own 16-lane row and arrive by
        // DPP row broadcast; only the finished pivot value N(s, jj) crosses rows (bpermute).
        const int jj = lane & 15;
        float2 nv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) nv[r] = make_float2(4 * g + r == jj ? 1.f : 0.f, 0.f);
        inverse_steps(nv, xd, g, jj, std::make_integer_sequence<int, 15>{});
        {
            char* ndb = S + offsetof(typename Smem<C>::Set, nd) + rb * 1024;
#pragma unroll
            for (int r = 0; r < 4; ++r)
                *reinterpret_cast<u32*>(ndb + blk_off(4 * g + r, jj)) = pack_bf16(nv[r].x, nv[r].y);
        }
    };

    auto produce2 = [&](int ch) {
        // inputs of the next chunk are fetched first, so their latency overlaps this phase
        if (ch + 1 < nchunks) load_p(ch + 1);
        produce2_blocks(ch);
    };

    // ---------------------------------------------------------------- consumer phases
    auto consume1 = [&](int ch) {          // Delta of chunk ch
        const char* S = set_off(ch & 1);
        const auto& st = sm.set[ch & 1];
        u32x4 sb[CBW][4];          // S as B fragments
#pragma unroll
        for (int w = 0; w < CBW; ++w)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) sb[w][kb] = bfrag(Sacc[w][kb], nsign);
        // all blocks of Kg S first (NRB * CBW independent accumulator chains)
        f32x4 R[NRB][CBW];
#pragma unroll
        for (int p = 0; p < NRB; ++p)
#pragma unroll
            for (int w = 0; w < CBW; ++w) R[p][w] = zero4();
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int p = 0; p < NRB; ++p) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, kg) + rm_frag(p * 16 + c, kb * 4 + g));
#pragma unroll
                for (int w = 0; w < CBW; ++w) R[p][w] = mfma(a, sb[w][kb], R[p][w]);
            }
        // R = beta (conj(V) - Kg S)
#pragma unroll
        for (int p = 0; p < NRB; ++p) {
            const float4 bt = *reinterpret_cast<const float4*>(&st.beta[p * 16 + 4 * g]);
            const float btr[4] = {bt.x, bt.y, bt.z, bt.w};
#pragma unroll
            for (int w = 0; w < CBW; ++w) {
                const int cb = CBW * wave + w;
                const bool col_ok = cb < ncb && n0 + cb * 8 + (c >> 1) < n;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const u32 word = vv[w][p][r >> 1];
                    const bool ok = col_ok && (ch * C + p * 16 + 4 * g + r) < T;
                    const float vx = ok ? flip((r & 1) ? bf_hi(word) : bf_lo(word), csign) : 0.f;
                    R[p][w][r] = btr[r] * (vx - R[p][w][r]);
                }
            }
        }
        // blocked forward substitution: Delta_p = N_pp (R_p + sum_{q<p} (-(D_beta L'))_pq Delta_q)
#pragma unroll
        for (int p = 0; p < NRB; ++p) {
#pragma unroll
            for (int q2 = 0; q2 < p; ++q2) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, lb) + (p * (p - 1) / 2 + q2) * 1024 + blk_frag(c, g));
#pragma unroll
                for (int w = 0; w < CBW; ++w) R[p][w] = mfma(a, db[w][q2], R[p][w]);
            }
            const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, nd) + p * 1024 + blk_frag(c, g));
#pragma unroll
            for (int w = 0; w < CBW; ++w) {
                const f32x4 d = mfma(a, bfrag(R[p][w], nsign), zero4());
                db[w][p] = bfrag(d, nsign);
            }
        }
    };

    TOUT* const go = static_cast<TOUT*>(args.o);
    auto consume2 = [&](int ch) {          // outputs and state update of chunk ch
        const char* S = set_off(ch & 1);
        const auto& st = sm.set[ch & 1];
        const int t0 = ch * C;
        u32x4 sb[CBW][4];          // S (still the chunk-start state) as B fragments
#pragma unroll
        for (int w = 0; w < CBW; ++w)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) sb[w][kb] = bfrag(Sacc[w][kb], nsign);
        // O^* = conj(Q)G S + tril(A) Delta for all blocks, then the state update -- all
        // independent accumulator chains, issued before any output is stored
        f32x4 O[NRB][CBW];
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
            for (int w = 0; w < CBW; ++w) O[rb][w] = zero4();
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, qg) + rm_frag(rb * 16 + c, kb * 4 + g));
#pragma unroll
                for (int w = 0; w < CBW; ++w) O[rb][w] = mfma(a, sb[w][kb], O[rb][w]);
            }
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
            for (int jb = 0; jb <= rb; ++jb) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(S + offsetof(typename Smem<C>::Set, aq) + (rb * (rb + 1) / 2 + jb) * 1024 + blk_frag(c, g));
#pragma unroll
                for (int w = 0; w < CBW; ++w) O[rb][w] = mfma(a, db[w][jb], O[rb][w]);
            }
        // S <- diag(g_C) (S + (K/G)^T Delta)
#pragma unroll
        for (int tb = 0; tb < NRB; ++tb)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                const int irow = kb * 16 + c;
                u32x4 a;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    a[r] = *reinterpret_cast<const u32*>(S + offsetof(typename Smem<C>::Set, ki) + rm_off(tb * 16 + 4 * g + r, irow));
#pragma unroll
                for (int w = 0; w < CBW; ++w) Sacc[w][kb] = mfma(a, db[w][tb], Sacc[w][kb]);
            }
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float2 gg = st.gc[kb * 16 + 4 * g + r];
#pragma unroll
                for (int w = 0; w < CBW; ++w) {
                    const float own = Sacc[w][kb][r];
                    const float oth = partner(own);
                    Sacc[w][kb][r] = gg.x * own + flip(gg.y, nsign) * oth;
                }
            }
        // o = conj(O^*).  Whole tiles go through this wave's LDS stage so that every lane
        // writes 16 contiguous bytes; a ragged tile is written element by element.
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            const bool full = (t0 + rb * 16 + 16 <= T) && (n0 + CBW * 8 * (wave + 1) <= n) && (n & 3) == 0;
            if (full) {
                constexpr int PITCH = CBW * 16 * static_cast<int>(sizeof(TOUT));   // bytes per row
                char* stg = reinterpret_cast<char*>(sm.ostage[wave]);
#pragma unroll
                for (int w = 0; w < CBW; ++w)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        *reinterpret_cast<TOUT*>(stg + (4 * g + r) * PITCH + ((w * 8 + (c >> 1)) * 2 + qp) * sizeof(TOUT)) =
                            to_out<TOUT>(flip(O[rb][w][r], csign));
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                constexpr int CPR = PITCH / 16;                  // 16-byte pieces per row
                char* obase = reinterpret_cast<char*>(go + 2 * (base_tn + static_cast<long>(t0 + rb * 16) * n + n0 + CBW * 8 * wave));
#pragma unroll
                for (int idx0 = 0; idx0 < 16 * CPR; idx0 += 64) {
                    const int idx = idx0 + lane;
                    if (16 * CPR % 64 == 0 || idx < 16 * CPR) {
                        const int row = idx / CPR, piece = idx % CPR;
                        *reinterpret_cast<u32x4*>(obase + static_cast<long>(row) * n * 2 * sizeof(TOUT) + piece * 16) =
                            *reinterpret_cast<const u32x4*>(stg + row * PITCH + piece * 16);
                    }
                }
                __builtin_amdgcn_wave_barrier();   // stage reads finish before the next tile's writes
            } else {
#pragma unroll
                for (int w = 0; w < CBW; ++w) {
                    const int cb = CBW * wave + w;
                    const int j = n0 + cb * 8 + (c >> 1);
                    if (cb < ncb && j < n) {
                        TOUT* const orow = go + 2 * (base_tn + static_cast<long>(t0 + rb * 16 + 4 * g) * n + j) + qp;
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (t0 + rb * 16 + 4 * g + r < T)
                                Elem<TOUT>::store(orow, 2L * r * n, flip(O[rb][w][r], csign));
                    }
                }
            }
        }
        if (ch + 1 < nchunks) load_v(ch + 1);
    };

    auto consume_gram = [&](int ch) {      // A blocks of chunk ch (consumer waves, set ch & 1)
        char* S = set_off(ch & 1);
        int units[3][2];
        const int nu = unit_list(wave, units);
        for (int u = 0; u < nu; ++u) {
            const int rb = units[u][0], jb = units[u][1];
            f32x4 accA[2];
            gram_unit(S, offsetof(typename Smem<C>::Set, qg), rb, jb, accA);
            char* aqb = S + offsetof(typename Smem<C>::Set, aq) + (rb * (rb + 1) / 2 + jb) * 1024;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int jl = h * 8 + (c >> 1);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int tl = 4 * g + r;
                    const float va = (jb < rb || jl <= tl) ? accA[h][r] : 0.f;
                    *reinterpret_cast<__bf16*>(aqb + blk_off(tl, jl) + 2 * qp) = static_cast<__bf16>(va);
                }
            }
        }
    };

    // ---------------------------------------------------------------- roles
    // The role test is wave-uniform and encloses each role's whole life (prologue, chunk
    // loop, epilogue), so each role keeps only its own registers live.  Both loops pass the
    // same sequence of workgroup barriers: two per chunk plus the producers' lead-in chunk.
    if (consumer) {
#pragma unroll
        for (int w = 0; w < CBW; ++w) {
            const int cb = CBW * wave + w;
            const int j = n0 + cb * 8 + (c >> 1);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = kb * 16 + 4 * g + r;
                    float x = 0.f;
                    if (args.S0 != nullptr) {   // uniform test; the load itself is unconditional
                        // (clamped index, masked by a multiply so that no load waits alone)
                        const float keep = (cb < ncb && j < n && i < m) ? 1.f : 0.f;
                        x = keep * args.S0[2 * (base_mn + static_cast<long>(min(i, m - 1)) * n + min(j, n - 1)) + qp];
                    }
                    Sacc[w][kb][r] = x;
                }
        }
        if (nchunks > 0) load_v(0);
        for (int ch = -1; ch < nchunks; ++ch) {
            if (ch >= 0) consume1(ch);
            __syncthreads();
            if (ch >= 0) consume2(ch);
            if (ch + 1 < nchunks) consume_gram(ch + 1);   // operands written in phase 1
            __syncthreads();
        }
        if (args.S_T != nullptr) {
#pragma unroll
            for (int w = 0; w < CBW; ++w) {
                const int cb = CBW * wave + w;
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
#define SFDA_PIPE_LAUNCH(C_, W_) \
    hipLaunchKernelGGL((chunk_pipe_kernel<TOUT, C_, W_>), grid, dim3(NTH), 0, st, a)
    const bool wide = L.slice > 32;
    switch (L.C) {
        case 16: if (wide) SFDA_PIPE_LAUNCH(16, 2); else SFDA_PIPE_LAUNCH(16, 1); break;
        case 32: if (wide) SFDA_PIPE_LAUNCH(32, 2); else SFDA_PIPE_LAUNCH(32, 1); break;
        case 64: if (wide) SFDA_PIPE_LAUNCH(64, 2); else SFDA_PIPE_LAUNCH(64, 1); break;
        default: return hipErrorInvalidValue;
    }
#undef SFDA_PIPE_LAUNCH
    return hipGetLastError();
}

}  // namespace pipe

hipError_t launch_chunk_bf16(const ChunkLaunch& L, hipStream_t st)
{
    return L.out_bf16 ? pipe::launch_t<uint16_t>(L, st) : pipe::launch_t<float>(L, st);
}

}  // namespace sfda
