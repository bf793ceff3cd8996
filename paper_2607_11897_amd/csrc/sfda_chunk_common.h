// Shared pieces of the fp32-path chunk kernels (forward scan, adjoint scan, per-chunk
// gradients): launch arguments, the LDS layout of one chunk's operands, and the two
// state-independent stages every one of them starts a chunk with (the scans follow them
// with the triangular inverse, inline in their kernel).
//
// Inside a chunk of C tokens (Thm 4.2 / Cor. 4.3 chunk-WY factors), with g_t the running
// product of the decays lambda_1 ... lambda_t (the diagonal of Gamma_t):
//   load   conj(Q) * G, conj(K) * G and K / G into LDS (the decay-scaled operands);
//   gram   L'[t, j] = k_t^* diag(g_t / g_j) k_j (j < t) and A[r, j] = q_r^* diag(g_r / g_j) k_j
//          (j <= r) on the matrix cores, packed in one C x C buffer.
#pragma once

#include "sfda_device.h"
#include "sfda_launch.h"

namespace sfda {

// ----------------------------------------------------------------- buffer loads

// Reads through a buffer resource: a read past the resource's size returns zero, so rows
// past the end of a sequence or a block need no mask, and a lane outside the valid columns
// passes an offset past every resource (OOR).  No select follows such a load, so the loads
// of a stage issue back to back and are waited on once (a masked load, whose value is
// pinned before the select, waits right after it is issued).
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t OOR = 0x80000000u;
__device__ __forceinline__ rsrc_t buf(const void* base, long bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000);
}
__device__ __forceinline__ float2 ld_c64(rsrc_t r, uint32_t off) {      // complex float32
    return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}
__device__ __forceinline__ float ld_f32(rsrc_t r, uint32_t off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
template <typename T> __device__ __forceinline__ float2 ld_cplx(rsrc_t r, uint32_t off);
template <> __device__ __forceinline__ float2 ld_cplx<float>(rsrc_t r, uint32_t off) { return ld_c64(r, off); }
template <> __device__ __forceinline__ float2 ld_cplx<uint16_t>(rsrc_t r, uint32_t off) {
    const uint32_t w = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
    return make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
}
template <typename T> __device__ __forceinline__ float ld_real(rsrc_t r, uint32_t off);
template <> __device__ __forceinline__ float ld_real<float>(rsrc_t r, uint32_t off) { return ld_f32(r, off); }
template <> __device__ __forceinline__ float ld_real<uint16_t>(rsrc_t r, uint32_t off) {
    return __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0)) << 16);
}


constexpr int MP = 64;            // key channels handled per workgroup (m is zero-padded)
constexpr int LDX = MP + 1;       // complex row stride of the C x MP operand arrays
constexpr int NTHR = 256;

struct ChunkArgs {
    const void *q, *k, *v, *alpha, *theta, *beta;
    const float* S0;     // adjoint scan: dL/dS_T (may be null)
    void* o;
    float* S_T;          // adjoint scan: dL/dS0
    int T, m, n, n_slices, slice;
    // GATED: alpha = amin + aspan sigmoid(a), theta = tmax tanh(b), beta = sigmoid(c),
    // k = k~ / (||k~|| + eps) from the pre-activations passed in alpha, theta, beta, k
    float amin, aspan, tmax, eps;
    // backward passes: per-chunk records [heads][chunks][m][n] (state entering the chunk,
    // or the adjoint of the state leaving it) and [heads][chunks * C][n] (Delta, or G_F)
    float* ck_state;
    float* ck_rows;
    const void* dO;      // adjoint scan: dL/do, o's dtype
    void* dv;            // adjoint scan: dL/dv, the inputs' dtype
    // write-decoupled forward: write directions r [B,H,T,m] complex and write strengths
    // [B,H,T] (beta then holds the erase strengths eta)
    const void* r;
    const void* wbeta;
    // segment forward (MODE 4): the transfer columns' outputs X_t = P_t^* q_t
    // [heads][T][m] and last transfer P [heads][m][m], complex fp32 (either may be null)
    float* xo;
    float* pend;
};

__device__ __forceinline__ float sigmoid_acc(float x) { return 1.f / (1.f + expf(-x)); }

// Four LDS entries at(r), r = 0..3, read on every lane -- each read issued before any is
// waited for -- then kept where keep(r) and zero elsewhere.  (A read made conditional, or
// pinned one at a time, is issued and waited for on its own.)
template <typename AT, typename KEEP>
__device__ __forceinline__ void lds_masked4(AT at, KEEP keep, float2 (&x)[4])
{
#pragma unroll
    for (int r = 0; r < 4; ++r) x[r] = at(r);
#pragma unroll
    for (int r = 0; r < 4; ++r) x[r] = pin(x[r]);
#pragma unroll
    for (int r = 0; r < 4; ++r) x[r] = keep(r) ? x[r] : make_float2(0.f, 0.f);
}

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

// the role-split scans (16-token chunks) keep N = (I + D_beta L')^{-1} apart from L' (two
// waves form it, so it cannot be written over L' while the other may still read L')
template <int C>
struct ChunkSmemPipe : ChunkSmem<C> {
    float2 nn[C * ChunkSmem<C>::LDG];        // N, strict lower triangle
};

// the write-decoupled forward also keeps R / G, the k-r and q-r Gram blocks and the write
// strengths
template <int C>
struct ChunkSmemDec : ChunkSmemPipe<C> {
    float2 ri[C * LDX];                      // r_t / g_t
    float2 g3[C * ChunkSmem<C>::LDG];        // packed: L'_kr (strict lower), A_qr^T (strict upper), A_qr diag
    float wb[C];                             // write strengths beta_t
};

// alpha, theta, beta, q and k of one thread's tokens, fetched a chunk ahead by a scan, as
// the loaded words (a bf16 value is converted where it is used, so the fetch is not waited
// on where it is issued); q, k take one word per complex bf16 value, two per complex fp32.
// The write-decoupled forward also fetches the write directions r and write strengths.
template <int C>
struct InPre {
    uint32_t a[C / 4], th[C / 4], b;
    uint32_t q[C / 4][2], k[C / 4][2];
    uint32_t r[C / 4][2], wb;
};
template <typename TIN> __device__ __forceinline__ uint32_t raw_word(const void* p, long e) {
    if constexpr (sizeof(TIN) == 2) return static_cast<const uint16_t*>(p)[e];
    else return __float_as_uint(static_cast<const float*>(p)[e]);
}
template <typename TIN> __device__ __forceinline__ float word_f(uint32_t w) {
    return __uint_as_float(sizeof(TIN) == 2 ? w << 16 : w);
}

template <typename TIN, int C, bool WIDE, bool DEC = false>
__device__ __forceinline__ void prefetch_inputs(const ChunkArgs& args, long bh, int t0, int tid, InPre<C>& pf)
{
    constexpr int SEG = C / 4;
    if (WIDE && tid >= NTHR) return;
    const int T = args.T, m = args.m;
    const long base_tm = bh * static_cast<long>(T) * m;
    const int i = tid & 63, seg = (tid >> 6) & 3;
#pragma unroll
    for (int u = 0; u < SEG; ++u) {
        const int t = t0 + seg * SEG + u;
        const long e = base_tm + static_cast<long>(min(t, T - 1)) * m + min(i, m - 1);
        pf.a[u] = raw_word<TIN>(args.alpha, e);
        pf.th[u] = raw_word<TIN>(args.theta, e);
        if constexpr (sizeof(TIN) == 2) {
            pf.q[u][0] = static_cast<const uint32_t*>(args.q)[e];
            pf.k[u][0] = static_cast<const uint32_t*>(args.k)[e];
        } else {
            const uint2 qw = static_cast<const uint2*>(args.q)[e], kw = static_cast<const uint2*>(args.k)[e];
            pf.q[u][0] = qw.x; pf.q[u][1] = qw.y;
            pf.k[u][0] = kw.x; pf.k[u][1] = kw.y;
        }
        if constexpr (DEC) {
            if constexpr (sizeof(TIN) == 2) {
                pf.r[u][0] = static_cast<const uint32_t*>(args.r)[e];
            } else {
                const uint2 rw = static_cast<const uint2*>(args.r)[e];
                pf.r[u][0] = rw.x; pf.r[u][1] = rw.y;
            }
        }
    }
    const long eb = bh * static_cast<long>(T) + min(t0 + (tid & (C - 1)), T - 1);
    pf.b = raw_word<TIN>(args.beta, eb);
    if constexpr (DEC) pf.wb = raw_word<TIN>(args.wbeta, eb);
}

// ----------------------------------------------------------------- load stage
// Thread (channel i = tid % 64, segment tid / 64) walks C / 4 consecutive tokens of the
// chunk starting at t0: running sums of log alpha and theta give g_t; the decay-scaled
// operands go to LDS.  Padding past T (and channels past m) are identity tokens.  With
// KEEP, g_t of the thread's tokens is returned in gkeep; with DEC (SM = ChunkSmemDec) the
// write directions become R / G and the write strengths are loaded too.  In a block wider
// than 256 threads (WIDE) only the first 256 work; every thread passes the barrier.  With
// PRE, alpha, theta and beta come from *pre (fetched a chunk ahead) and q, k are requested
// before the running sums, so their latency overlaps the sums and the barrier.
template <typename TIN, int C, bool GATED, bool KEEP = false, bool DEC = false, typename SM = ChunkSmem<C>,
          bool WIDE = false, bool PRE = false>
__device__ __forceinline__ void stage_load(SM& sm, const ChunkArgs& args, long bh,
                                           int t0, int tid, float2 (&gkeep)[C / 4],
                                           const InPre<C>* pre = nullptr)
{
    const bool worker = !WIDE || tid < NTHR;
    constexpr int SEG = C / 4;
    const TIN* __restrict__ gq = static_cast<const TIN*>(args.q);
    const TIN* __restrict__ gk = static_cast<const TIN*>(args.k);
    const TIN* __restrict__ ga = static_cast<const TIN*>(args.alpha);
    const TIN* __restrict__ gth = static_cast<const TIN*>(args.theta);
    const TIN* __restrict__ gb = static_cast<const TIN*>(args.beta);
    const int T = args.T, m = args.m;
    const long base_tm = bh * static_cast<long>(T) * m;

    const int i = tid & 63;
    const int seg = (tid >> 6) & 3;
    // (without PRE: alpha, theta, q, k through resources over this chunk's rows)
    const long rbytes = static_cast<long>(min(T - t0, C)) * m * sizeof(TIN);
    const rsrc_t ra = buf(ga + base_tm + static_cast<long>(t0) * m, rbytes);
    const rsrc_t rt = buf(gth + base_tm + static_cast<long>(t0) * m, rbytes);
    const rsrc_t rq = buf(gq + 2 * (base_tm + static_cast<long>(t0) * m), 2 * rbytes);
    const rsrc_t rk = buf(gk + 2 * (base_tm + static_cast<long>(t0) * m), 2 * rbytes);
    float la[SEG], ph[SEG];
    float sa = 0.f, sp = 0.f;
    float2 qpre[PRE ? SEG : 1], kpre[PRE ? SEG : 1];
    if constexpr (PRE) {            // q, k from the chunk-ahead fetch
#pragma unroll
        for (int u = 0; u < SEG; ++u) {
            if constexpr (sizeof(TIN) == 2) {
                qpre[u] = make_float2(__uint_as_float(pre->q[u][0] << 16), __uint_as_float(pre->q[u][0] & 0xFFFF0000u));
                kpre[u] = make_float2(__uint_as_float(pre->k[u][0] << 16), __uint_as_float(pre->k[u][0] & 0xFFFF0000u));
            } else {
                qpre[u] = make_float2(__uint_as_float(pre->q[u][0]), __uint_as_float(pre->q[u][1]));
                kpre[u] = make_float2(__uint_as_float(pre->k[u][0]), __uint_as_float(pre->k[u][1]));
            }
        }
    }
    if (worker) {
#pragma unroll
    for (int u = 0; u < SEG; ++u) {
        const int t = t0 + seg * SEG + u;
        const bool ok = t < T && i < m;
        const long e = base_tm + static_cast<long>(min(t, T - 1)) * m + min(i, m - 1);
        float a_ld, th;
        float a;
        if constexpr (PRE) {
            a_ld = pin(word_f<TIN>(pre->a[u]));
            th = masked(ok, word_f<TIN>(pre->th[u]));
            a = ok ? a_ld : 1.f;
        } else {
            // buffer reads, zero past T and past m: no pin, so they issue back to back
            const uint32_t off = i < m ? static_cast<uint32_t>((t - t0) * m + i) * static_cast<uint32_t>(sizeof(TIN)) : OOR;
            a_ld = ld_real<TIN>(ra, off);
            th = ld_real<TIN>(rt, off);
            a = a_ld + (ok ? 0.f : 1.f);          // the identity token's alpha is 1
        }
        if constexpr (GATED) {      // padding stays the identity token (alpha = 1, theta = 0)
            a = ok ? args.amin + args.aspan * sigmoid_acc(a_ld) : 1.f;
            th = ok ? args.tmax * tanhf(th) : 0.f;
        }
        sa += __logf(a);
        // phase in revolutions, reduced to [0, 1) at every token, so that the sine and
        // cosine below see a small argument whatever theta is
        sp = __builtin_amdgcn_fractf(__builtin_fmaf(th, 0.15915494309189535f, sp));
        la[u] = sa;
        ph[u] = sp;
    }
    sm.sega[seg][i] = sa;
    sm.segp[seg][i] = sp;
    }
    if (worker) {
        const int tb = t0 + (tid & (C - 1));
        float bv;
        if constexpr (PRE) bv = word_f<TIN>(pre->b);
        else bv = Elem<TIN>::load(gb, bh * static_cast<long>(T) + min(tb, T - 1));
        if constexpr (GATED) bv = sigmoid_acc(bv);
        if (tid < C) sm.beta[tid] = masked(tb < T, bv);
        if constexpr (DEC) {
            float wv;
            if constexpr (PRE) wv = word_f<TIN>(pre->wb);
            else wv = Elem<TIN>::load(static_cast<const TIN*>(args.wbeta), bh * static_cast<long>(T) + min(tb, T - 1));
            if (tid < C) sm.wb[tid] = masked(tb < T, wv);
        }
    }
    __syncthreads();
    if (!worker) return;
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
        // 1 / |g_t| stays finite while the chunk's decay so far is at least 2^-126; past
        // that the operand is NaN, so the chunk's outputs from here on and every later
        // state are NaN rather than silently wrong
        const float ei = A >= -87.3365447f ? __expf(-A) : __builtin_nanf("");
        const float sn = __builtin_amdgcn_sinf(Ph), cs = __builtin_amdgcn_cosf(Ph);   // Ph in revolutions
        const float gr = e * cs, gi = e * sn;        // g_t
        const float hr = ei * cs, hi = -ei * sn;     // 1 / g_t
        if constexpr (KEEP) gkeep[u] = make_float2(gr, gi);
        const bool ok = t < T && i < m;
        const long e2 = base_tm + static_cast<long>(min(t, T - 1)) * m + min(i, m - 1);
        float2 qq, kk;
        if constexpr (PRE) {
            qq = masked(ok, qpre[u]);
            kk = masked(ok, kpre[u]);
        } else {                                     // zero past T and past m
            const uint32_t off = i < m ? static_cast<uint32_t>(tl * m + i) * static_cast<uint32_t>(2 * sizeof(TIN)) : OOR;
            qq = ld_cplx<TIN>(rq, off);
            kk = ld_cplx<TIN>(rk, off);
        }
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
        if constexpr (DEC) {
            float2 rr;
            if constexpr (PRE) {
                if constexpr (sizeof(TIN) == 2)
                    rr = make_float2(__uint_as_float(pre->r[u][0] << 16), __uint_as_float(pre->r[u][0] & 0xFFFF0000u));
                else
                    rr = make_float2(__uint_as_float(pre->r[u][0]), __uint_as_float(pre->r[u][1]));
            } else {
                rr = Elem<TIN>::load2(static_cast<const TIN*>(args.r), e2);
            }
            rr = masked(ok, rr);
            sm.ri[tl * LDX + i] = make_float2(rr.x * hr - rr.y * hi, rr.x * hi + rr.y * hr);
        }
        if (tl == C - 1) sm.gc[i] = make_float2(gr, gi);
    }
}

// ----------------------------------------------------------------- gram stage
// L' (strict lower, at g2[t][j]) and, with WANT_A, A (A[r][j] for j < r at g2[j][r], the
// diagonal at g2[r][r]).  Reads qg, kg, ki; the caller synchronises before and after.
// With ROP (SM = ChunkSmemDec) the right operand is R / G instead of K / G and the blocks
// (L'_kr, A_qr) go to g3.
template <int P, int C, bool WANT_A, bool ROP = false, typename SM = ChunkSmem<C>, int NW = 4>
__device__ __forceinline__ void stage_gram(SM& sm, int tid)
{
    constexpr int NRB = C / 16;
    constexpr int LDG = ChunkSmem<C>::LDG;
    constexpr int NCB = C / 8;                       // real column blocks of C x C
    constexpr int NT1 = NRB * (NRB + 1);             // causal tiles per matrix
    const int lane = tid & 63, wave = tid >> 6;
    const int c = lane & 15, g = lane >> 4, qp = lane & 1;
    float* g2f;
    const float2* Yop;
    if constexpr (ROP) {
        g2f = reinterpret_cast<float*>(sm.g3);
        Yop = sm.ri;
    } else {
        g2f = reinterpret_cast<float*>(sm.g2);
        Yop = sm.ki;
    }
    for (int tile = wave; tile < (WANT_A ? 2 : 1) * NT1; tile += NW) {
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
                const float2 y = Yop[jcol * LDX + i];     // B(i, j) = (K/G)^T (or (R/G)^T)
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

}  // namespace sfda
