// Segment-parallel scan helpers: a long sequence of a head is cut into G segments that
// run as independent heads of the chunk kernel; the state entering each segment then
// follows from the affine law of a segment (Thm 4.4: the state after a stretch of tokens
// is P S_in + B, with P the product of the stretch's transitions A_t and B its write from
// the zero state) composed along the segments (Lemma A.2):
//   S_in[0] = S0,   S_in[g + 1] = P_g S_in[g] + B_g,   S_T = S_in[G].
// P_g is the chunk kernel's final state for S0 = I and v = 0 (then every B_t = 0), B_g its
// final state for S0 = 0.  The outputs follow from the same law token by token: with P_t the
// product of the segment's transitions up to token t and o0_t the output of the zero-state
// pass, o_t = (P_t S_in + B_t)^* q_t = o0_t + S_in^* X_t, X_t = P_t^* q_t, and X_t is the
// output of the S0 = I pass (its n = m columns).  This file holds the identity fill for that
// pass, the fold and the join o_t += S_in^* X_t.
#include <stdint.h>

#include "sfda_device.h"
#include "sfda_launch.h"

namespace sfda {
namespace seg {

constexpr int NT = 256;
constexpr int MP = 64;      // state rows (m <= 64)
constexpr int CB = 8;       // value columns per workgroup in the fold
constexpr int CPT = CB / 4; // of them per thread

// P[s] = I (m x m complex), s < count
__global__ __launch_bounds__(NT) void identity_kernel(float* P, long count, int m)
{
    const long mm = static_cast<long>(m) * m;
    const long total = count * mm;
    for (long e = blockIdx.x * static_cast<long>(NT) + threadIdx.x; e < total;
         e += static_cast<long>(gridDim.x) * NT) {
        const long r = e % mm;
        const int i = static_cast<int>(r / m), j = static_cast<int>(r % m);
        reinterpret_cast<float2*>(P)[e] = make_float2(i == j ? 1.f : 0.f, 0.f);
    }
}

// One workgroup per (head, block of CB value columns).  Column j of the state only mixes
// with column j, so a block of columns runs the fold on its own, held in LDS.
// P: [heads * G][m][m], Bs, Sin: [heads * G][m][n], S0, S_T: [heads][m][n] (complex
// float32; S0 may be null = zero state, S_T may be null).
__global__ __launch_bounds__(NT) void fold_kernel(const float* __restrict__ P,
                                                  const float* __restrict__ Bs,
                                                  float* __restrict__ Sin,
                                                  const float* __restrict__ S0,
                                                  float* __restrict__ S_T,
                                                  int G, int m, int n, int ncb)
{
    __shared__ float2 S[MP][CB];
    __shared__ float2 Ps[MP][MP + 1];     // P_g, rows padded against bank conflicts
    const long h = blockIdx.x / ncb;
    const int j0 = static_cast<int>(blockIdx.x - h * ncb) * CB;
    const int tid = threadIdx.x;
    const int i = tid >> 2;             // state row
    const int jq = (tid & 3) * CPT;     // first of this thread's CPT columns in the block
    const long mn = static_cast<long>(m) * n;
    const float2* P2 = reinterpret_cast<const float2*>(P);
    const float2* B2 = reinterpret_cast<const float2*>(Bs);
    float2* Sin2 = reinterpret_cast<float2*>(Sin);

    auto col_ok = [&](int c) { return j0 + jq + c < n; };
    float2 s[CPT];
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
        s[c] = make_float2(0.f, 0.f);
        if (S0 != nullptr && i < m && col_ok(c))
            s[c] = reinterpret_cast<const float2*>(S0)[h * mn + static_cast<long>(i) * n + j0 + jq + c];
        S[i][jq + c] = s[c];
    }
    // P_g is fetched a segment ahead into registers (coalesced: element e = r * m + l of the
    // m x m block, NPF per thread), so its load overlaps the products of the segment before
    constexpr int NPF = MP * MP / NT;
    float2 pf[NPF];
    auto fetch_p = [&](long seg) {
        const float2* pg = P2 + seg * static_cast<long>(m) * m;
#pragma unroll
        for (int u = 0; u < NPF; ++u) {
            const int e = u * NT + tid;
            pf[u] = e < m * m ? pg[e] : make_float2(0.f, 0.f);
        }
    };
    fetch_p(h * G);
    __syncthreads();
    for (int gi = 0; gi < G; ++gi) {
        const long seg = h * G + gi;
        // the state entering segment gi
        if (i < m) {
#pragma unroll
            for (int c = 0; c < CPT; ++c)
                if (col_ok(c)) Sin2[seg * mn + static_cast<long>(i) * n + j0 + jq + c] = s[c];
        }
#pragma unroll
        for (int u = 0; u < NPF; ++u) {
            const int e = u * NT + tid;
            if (e < m * m) Ps[e / m][e % m] = pf[u];
        }
        __syncthreads();
        if (gi + 1 < G) fetch_p(seg + 1);
        // row i of P_gi S + B_gi
        float2 acc[CPT];
#pragma unroll
        for (int c = 0; c < CPT; ++c) acc[c] = make_float2(0.f, 0.f);
        if (i < m) {
            for (int l = 0; l < m; ++l) {
                const float2 p = Ps[i][l];
#pragma unroll
                for (int c = 0; c < CPT; ++c) {
                    const float2 x = S[l][jq + c];
                    acc[c].x = __builtin_fmaf(p.x, x.x, __builtin_fmaf(-p.y, x.y, acc[c].x));
                    acc[c].y = __builtin_fmaf(p.x, x.y, __builtin_fmaf(p.y, x.x, acc[c].y));
                }
            }
#pragma unroll
            for (int c = 0; c < CPT; ++c) {
                if (!col_ok(c)) continue;
                const float2 b = B2[seg * mn + static_cast<long>(i) * n + j0 + jq + c];
                acc[c].x += b.x;
                acc[c].y += b.y;
            }
        }
        __syncthreads();                // every row of S and of P_gi read
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            s[c] = acc[c];
            S[i][jq + c] = acc[c];
        }
        __syncthreads();
    }
    if (S_T != nullptr && i < m) {
#pragma unroll
        for (int c = 0; c < CPT; ++c)
            if (col_ok(c)) reinterpret_cast<float2*>(S_T)[h * mn + static_cast<long>(i) * n + j0 + jq + c] = s[c];
    }
}

// o[s][t][j] += sum_l conj(Sin[s][l][j]) X[s][t][l] for segment s, token t < Ts, column
// j < n (X: [segs][Ts][m], Sin: [segs][m][n] complex float32; o: [segs][Ts][n] complex TOUT,
// holding the zero-state outputs).  One workgroup (four waves) per (segment, 64 tokens, 64
// columns): the block's X rows and conj(Sin) columns in LDS, the product on fp32 matrix
// cores as complex 16 x 16 tiles (a 16-token x 8-column tile per MFMA accumulator, K over
// the m channels in blocks of 16), eight tiles per wave.
constexpr int JT = 64;      // tokens per join workgroup
constexpr int JC = 64;      // value columns per join workgroup
template <typename TOUT>
__global__ __launch_bounds__(NT) void join_kernel(const float* __restrict__ X,
                                                  const float* __restrict__ Sin,
                                                  TOUT* __restrict__ o, int Ts, int m, int n,
                                                  int ntb, int ncb)
{
    __shared__ float2 Xs[JT][MP + 1];
    __shared__ float2 Ss[MP][JC + 1];
    const long blocks_per_seg = static_cast<long>(ntb) * ncb;
    const long s = blockIdx.x / blocks_per_seg;
    const int rem = static_cast<int>(blockIdx.x - s * blocks_per_seg);
    const int t0 = (rem / ncb) * JT, j0 = (rem % ncb) * JC;
    const int tid = threadIdx.x;
    const float2* X2 = reinterpret_cast<const float2*>(X) + s * Ts * static_cast<long>(m);
    const float2* S2 = reinterpret_cast<const float2*>(Sin) + s * static_cast<long>(m) * n;
    // every load of the block requested before the first LDS write
    constexpr int LU = JT * MP / NT;
    static_assert(JT * MP % NT == 0 && MP * JC == JT * MP, "whole steps");
    float2 xr[LU], sr[LU];
#pragma unroll
    for (int u = 0; u < LU; ++u) {
        const int e = u * NT + tid;
        const int tt = e / MP, l = e % MP;
        xr[u] = (t0 + tt < Ts && l < m) ? X2[static_cast<long>(t0 + tt) * m + l] : make_float2(0.f, 0.f);
        const int l2 = e / JC, jj = e % JC;
        sr[u] = (l2 < m && j0 + jj < n) ? S2[static_cast<long>(l2) * n + j0 + jj] : make_float2(0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < LU; ++u) {
        const int e = u * NT + tid;
        Xs[e / MP][e % MP] = xr[u];
        Ss[e / JC][e % JC] = make_float2(sr[u].x, -sr[u].y);
    }
    __syncthreads();
    const int lane = tid & 63, wave = tid >> 6;
    const int c = lane & 15, g = lane >> 4, qp = lane & 1;
    const int nkb = (m + 15) / 16;
    // wave w: token tile w (16 tokens), the eight column tiles (8 complex columns each)
    f32x4 acc[8];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) acc[ct] = zero4();
    for (int kb = 0; kb < nkb; ++kb) {
        Frag8 a;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float2 x = Xs[wave * 16 + c][kb * 16 + 4 * g + r];
            a.v[2 * r] = x.x;
            a.v[2 * r + 1] = x.y;
        }
#pragma unroll
        for (int ct = 0; ct < 8; ++ct) {
            Frag8 b;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float2 y = Ss[kb * 16 + 4 * g + r][ct * 8 + (c >> 1)];
                bpair(b, r, y.x, y.y, qp);
            }
            mma<PREC_F32>(acc[ct], a, b);
        }
    }
    // lane (c, g) holds part qp of o[t = 4g + r][column c / 2] of each tile: the block goes
    // through LDS (over the X rows, read by now) so that the read-modify-write of o runs
    // row-contiguous, one complex element per lane and step
    __syncthreads();
    float* Os = reinterpret_cast<float*>(&Xs[0][0]);
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r)
            Os[2 * ((wave * 16 + 4 * g + r) * (MP + 1) + ct * 8 + (c >> 1)) + qp] = acc[ct][r];
    __syncthreads();
    constexpr int OU = JT * JC / NT;
    float2 z[OU];
#pragma unroll
    for (int u = 0; u < OU; ++u) {
        const int e = u * NT + tid;
        const int t = t0 + e / JC, j = j0 + e % JC;
        z[u] = (t < Ts && j < n) ? Elem<TOUT>::load2(o, (s * Ts + t) * static_cast<long>(n) + j)
                                 : make_float2(0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < OU; ++u) {
        const int e = u * NT + tid;
        const int tt = e / JC, jj = e % JC;
        const int t = t0 + tt, j = j0 + jj;
        if (t >= Ts || j >= n) continue;
        const float2 d = Xs[tt][jj];
        Elem<TOUT>::store2(o, (s * Ts + t) * static_cast<long>(n) + j, z[u].x + d.x, z[u].y + d.y);
    }
}

}  // namespace seg

hipError_t launch_join(const float* X, const float* Sin, void* o, bool out_bf16, long segs,
                       int Ts, int m, int n, hipStream_t st)
{
    const int ntb = (Ts + seg::JT - 1) / seg::JT, ncb = (n + seg::JC - 1) / seg::JC;
    const dim3 grid(static_cast<unsigned>(segs * ntb * ncb));
    if (out_bf16)
        hipLaunchKernelGGL(seg::join_kernel<uint16_t>, grid, dim3(seg::NT), 0, st, X, Sin,
                           static_cast<uint16_t*>(o), Ts, m, n, ntb, ncb);
    else
        hipLaunchKernelGGL(seg::join_kernel<float>, grid, dim3(seg::NT), 0, st, X, Sin,
                           static_cast<float*>(o), Ts, m, n, ntb, ncb);
    return hipGetLastError();
}

hipError_t launch_identity(float* P, long count, int m, hipStream_t st)
{
    const long total = count * m * m;
    const long blocks = (total + seg::NT - 1) / seg::NT;
    const unsigned grid = static_cast<unsigned>(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096);
    hipLaunchKernelGGL(seg::identity_kernel, dim3(grid), dim3(seg::NT), 0, st, P, count, m);
    return hipGetLastError();
}

hipError_t launch_fold(const float* P, const float* Bs, float* Sin, const float* S0, float* S_T,
                       long heads, int G, int m, int n, hipStream_t st)
{
    const int ncb = (n + seg::CB - 1) / seg::CB;
    const dim3 grid(static_cast<unsigned>(heads * ncb));
    hipLaunchKernelGGL(seg::fold_kernel, grid, dim3(seg::NT), 0, st, P, Bs, Sin, S0, S_T, G, m, n, ncb);
    return hipGetLastError();
}

}  // namespace sfda
