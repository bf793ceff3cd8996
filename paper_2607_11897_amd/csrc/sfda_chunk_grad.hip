// Per-chunk gradient pass of the SFDA backward: one workgroup per (head, chunk), all
// chunks in parallel.  The two scans before it record, for every chunk, the state S
// entering it, dL/dS of the state leaving it (G), Delta and G_F (the adjoint of the solve's
// right-hand side); with those the chunk's gradients are local.
//
// Chunk relations (Thm 4.2 / Cor. 4.3 factors, Thm 4.4 transfer, Thm 4.5 outputs; the
// forward kernel's notation):
//   E = conj(V) - (conj(K) G) S,  (I + D_beta L') Delta = D_beta E,  Delta = D_beta H,
//   O^* = (conj(Q) G) S + tril(A) Delta,  S_out = diag(g_C) S + Y'^T Delta,  Y' = (K/G) diag(g_C)
// with L' = strict_tril((conj(K) G)(K/G)^T) and A = tril((conj(Q) G)(K/G)^T).  For a real
// loss, with the adjoint G_R = conj(dL/do) of O^* and G_E = D_beta G_F:
//   H       = E - L' Delta                     (the pre-beta innovation of each token)
//   dbeta_t = Re sum_c conj(G_F[t, c]) H[t, c]
//   G_A     = tril(G_R Delta^*),   G_L' = D_beta strict_tril(-G_F Delta^*)
//   G_Qg    = G_R S^* + G_A conj(K/G)                    (adjoint of conj(Q) G)
//   G_Kg    = -G_E S^* + G_L' conj(K/G)                  (adjoint of conj(K) G)
//   G_Ki    = conj(Delta) G^T diag(conj(g_C)) + G_L'^T conj(conj(K) G) + G_A^T conj(conj(Q) G)
//   G_gC    = rowsum(G * conj(S)) + colsum(conj(Delta) G^T * conj(K/G))
// and elementwise per token and channel (g the running decay product):
//   dq = g conj(G_Qg),   dk = g conj(G_Kg) + conj(1/g) G_Ki,
//   dL/dg = q G_Qg + k G_Kg - conj(k / g^2) G_Ki  (+ G_gC at the chunk's last token),
//   z = log g = sum(log alpha) + i sum(theta):  dL/dz = conj(g) dL/dg, and the sums turn
//   into suffix sums over the chunk: dalpha = suffix(Re dL/dz) / alpha, dtheta = suffix(Im).
// Gradients of a complex variable are dL/dRe + i dL/dIm.
//
// Products over the value dimension read their operands straight from the records (global
// memory, one 32-byte row piece per lane and K-block); products over tokens read the
// decay-scaled operands from LDS.  The C x C gradients G_L' and G_A share one LDS block
// (G_L' strict lower, G_A^T upper with the diagonal).
#include "sfda_chunk_common.h"

namespace sfda {

constexpr int GW = 8;        // waves per workgroup: two per SIMD, to hide the record loads' latency

struct GradArgs {
    ChunkArgs in;                          // q, k, v, alpha, theta, beta, T, m, n
    const void* dO;
    const float *S_rec, *G_rec, *D_rows, *F_rows;
    void *dq, *dk, *dalpha, *dtheta, *dbeta;
};

template <int P, typename TIN, typename TOUT, int C>
__global__ __launch_bounds__(GW * 64, C <= 32 ? 4 : 2) void grad_kernel(GradArgs A)
{
    constexpr int NRB = C / 16;
    constexpr int SEG = C / 4;
    constexpr int LDG = ChunkSmem<C>::LDG;
    constexpr int NCT = NRB * (2 * MP / 16);        // C x m output tiles (16 tokens x 8 channels)
    constexpr int NT1 = NRB * (NRB + 1);            // causal tiles of a C x C matrix
    __shared__ ChunkSmem<C> sm;
    __shared__ float dbeta_part[GW][C];             // per-wave shares of dbeta
    __shared__ float ggc[2 * MP];                   // dL/dg_C (complex)

    const ChunkArgs& args = A.in;
    const int T = args.T, m = args.m, n = args.n;
    const int nchunks = (T + C - 1) / C;
    const long bh = blockIdx.x / nchunks;
    const int ch = static_cast<int>(blockIdx.x - bh * nchunks);
    const int t0 = ch * C;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int c = lane & 15, g = lane >> 4, qp = lane & 1;
    const int nkb = (n + 15) / 16;                  // K-blocks over the value columns
    const int ncbn = (n + 7) / 8;                   // 8-column blocks of the value columns

    const float2* Srec = reinterpret_cast<const float2*>(A.S_rec) + (bh * nchunks + ch) * static_cast<long>(m) * n;
    const float2* Grec = reinterpret_cast<const float2*>(A.G_rec) + (bh * nchunks + ch) * static_cast<long>(m) * n;
    const float2* Drow = reinterpret_cast<const float2*>(A.D_rows) + (bh * nchunks * static_cast<long>(C) + t0) * n;
    const float2* Frow = reinterpret_cast<const float2*>(A.F_rows) + (bh * nchunks * static_cast<long>(C) + t0) * n;
    const TOUT* gdO = static_cast<const TOUT*>(A.dO);
    const TIN* gv = static_cast<const TIN*>(args.v);
    const long base_tn = bh * static_cast<long>(T) * n;
    const long base_tm = bh * static_cast<long>(T) * m;

    // record element (row, column) of a [rows][n] block, zero outside
    auto rec = [&](const float2* p, int row, int rows, int col) {
        const bool ok = row < rows && col < n;
        return masked(ok, p[static_cast<long>(min(row, rows - 1)) * n + min(col, n - 1)]);
    };
    // G_R = conj(dL/do) at chunk row tl, column col
    auto grad_out = [&](int tl, int col) {
        const int t = t0 + tl;
        const bool ok = t < T && col < n;
        float2 x = masked(ok, Elem<TOUT>::load2(gdO, base_tn + static_cast<long>(min(t, T - 1)) * n + min(col, n - 1)));
        return make_float2(x.x, -x.y);
    };
    // Four consecutive columns col0 .. col0 + 3 (col0 a multiple of 4) of one row: with n a
    // multiple of 4 the group is wholly inside or outside the row and 32-byte aligned, and a
    // lane fetches it with 16-byte loads (a wave touches 16 rows x 64 bytes per load instead
    // of 64 scattered 8-byte pieces); otherwise element by element.
    const bool vec4 = (n & 3) == 0;
    auto rec4 = [&](const float2* p, int row, int rows, int col0, float2 (&x)[4]) {
        if (vec4) {
            const bool ok = row < rows && col0 < n;
            const float4* q4 = reinterpret_cast<const float4*>(p + static_cast<long>(min(row, rows - 1)) * n + min(col0, n - 4));
            const float4 a = q4[0], b = q4[1];
            x[0] = masked(ok, make_float2(a.x, a.y));
            x[1] = masked(ok, make_float2(a.z, a.w));
            x[2] = masked(ok, make_float2(b.x, b.y));
            x[3] = masked(ok, make_float2(b.z, b.w));
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) x[r] = rec(p, row, rows, col0 + r);
        }
    };
    auto grad_out4 = [&](int tl, int col0, float2 (&x)[4]) {
        if (vec4) {
            const int t = t0 + tl;
            const bool ok = t < T && col0 < n;
            const long e = base_tn + static_cast<long>(min(t, T - 1)) * n + min(col0, n - 4);
            float2 y[4];
            if constexpr (sizeof(TOUT) == 4) {
                const float4* q4 = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(gdO) + 2 * e);
                const float4 a = q4[0], b = q4[1];
                y[0] = make_float2(a.x, a.y); y[1] = make_float2(a.z, a.w);
                y[2] = make_float2(b.x, b.y); y[3] = make_float2(b.z, b.w);
            } else {
                const uint4 w = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(gdO) + 2 * e);
                const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    y[r] = make_float2(__uint_as_float(ws[r] << 16), __uint_as_float(ws[r] & 0xFFFF0000u));
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float2 z = masked(ok, y[r]);
                x[r] = make_float2(z.x, -z.y);
            }
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) x[r] = grad_out(tl, col0 + r);
        }
    };

    // (the load stage and the elementwise stage work on the first 256 threads; the latter
    // forms g again rather than holding it in registers through the whole kernel)
    {
        // every input load of the stage in flight at once: alpha, theta, beta, then q, k
        InPre<C> pf;
        prefetch_inputs<TIN, C, true>(args, bh, t0, tid, pf);
        float2 gkeep[SEG];
        stage_load<TIN, C, false, false, false, ChunkSmem<C>, true, true>(sm, args, bh, t0, tid, gkeep, &pf);
    }
    // dL/dg_C, first part: sum over columns of G * conj(S), one state row per 8 threads
    {
        const int i = tid >> 3, part = tid & 7;
        float2 acc = make_float2(0.f, 0.f);
        for (int c0 = 0; c0 < n; c0 += 64) {
            float2 gs[8], sv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                gs[u] = rec(Grec, i, m, c0 + part + 8 * u);
                sv[u] = rec(Srec, i, m, c0 + part + 8 * u);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                acc.x += gs[u].x * sv[u].x + gs[u].y * sv[u].y;
                acc.y += gs[u].y * sv[u].x - gs[u].x * sv[u].y;
            }
        }
#pragma unroll
        for (int sh = 1; sh < 8; sh <<= 1) {
            acc.x += __shfl_xor(acc.x, sh);
            acc.y += __shfl_xor(acc.y, sh);
        }
        if (part == 0) {
            ggc[2 * i] = acc.x;
            ggc[2 * i + 1] = acc.y;
        }
    }
    __syncthreads();
    stage_gram<P, C, false, false, ChunkSmem<C>, GW>(sm, tid);   // L'
    __syncthreads();

    // ================================================================ H = E - L' Delta, dbeta
    // (each wave sums its column blocks in registers; the per-wave shares are added in a
    // fixed order at the end, so no atomics are needed)
    float dacc[NRB][4];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 4; ++r) dacc[rb][r] = 0.f;
    for (int cb = wave; cb < ncbn; cb += GW) {
        const int j = cb * 8 + (c >> 1);
        Frag8 sbf[MP / 16];                            // S, K = state row
#pragma unroll
        for (int kb = 0; kb < MP / 16; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float2 y = rec(Srec, kb * 16 + 4 * g + r, m, j);
                bpair(sbf[kb], r, y.x, y.y, qp);
            }
        Frag8 dbf[NRB];                                // Delta, K = token
#pragma unroll
        for (int kb = 0; kb < NRB; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float2 y = rec(Drow, kb * 16 + 4 * g + r, C, j);
                bpair(dbf[kb], r, y.x, y.y, qp);
            }
        float vpart[NRB][4], fpart[NRB][4];            // this lane's parts of conj(V) and G_F
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tl = rb * 16 + 4 * g + r;
                const int t = t0 + tl;
                const bool ok = t < T && j < n;
                float2 vv = make_float2(0.f, 0.f);
                if (gv != nullptr)
                    vv = Elem<TIN>::load2(gv, base_tn + static_cast<long>(min(t, T - 1)) * n + min(j, n - 1));
                vv = masked(ok, vv);
                vpart[rb][r] = qp ? -vv.y : vv.x;
                const float2 f = rec(Frow, tl, C, j);
                fpart[rb][r] = qp ? f.y : f.x;
            }
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            const int row = rb * 16 + c;
            f32x4 pw = zero4();                        // (conj(K) G) S + L' Delta
#pragma unroll
            for (int kb = 0; kb < MP / 16; ++kb) {
                Frag8 a;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float2 x = sm.kg[row * LDX + kb * 16 + 4 * g + r];
                    a.v[2 * r] = x.x;
                    a.v[2 * r + 1] = x.y;
                }
                mma<P>(pw, a, sbf[kb]);
            }
#pragma unroll
            for (int kb = 0; kb <= rb; ++kb) {
                Frag8 a;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int jt = kb * 16 + 4 * g + r;
                    const float2 x = masked(jt < row, pin(sm.g2[row * LDG + jt]));
                    a.v[2 * r] = x.x;
                    a.v[2 * r + 1] = x.y;
                }
                mma<P>(pw, a, dbf[kb]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float h = vpart[rb][r] - pw[r];                  // H, this lane's part
                float prod = fpart[rb][r] * h;                         // Re(conj(G_F) H) share
                prod += __shfl_xor(prod, 1);
                prod += __shfl_xor(prod, 2);
                prod += __shfl_xor(prod, 4);
                prod += __shfl_xor(prod, 8);
                dacc[rb][r] += prod;
            }
        }
    }
    if (c == 0) {
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
            for (int r = 0; r < 4; ++r) dbeta_part[wave][rb * 16 + 4 * g + r] = dacc[rb][r];
    }
    __syncthreads();                                   // every read of L' done

    // ================================================================ G_A, G_L' (into g2)
    {
        float* g2f = reinterpret_cast<float*>(sm.g2);
        for (int tile = wave; tile < 2 * NT1; tile += GW) {
            const int mat = tile / NT1;                // 0: G_N from G_F, 1: G_A from G_R
            int rem = tile - mat * NT1, rb = 0;
            while (rem >= min(C / 8, 2 * rb + 2)) { rem -= min(C / 8, 2 * rb + 2); ++rb; }
            const int row = rb * 16 + c;
            const int jcol = rem * 8 + (c >> 1);
            f32x4 acc = zero4();
            for (int k0 = 0; k0 < nkb; k0 += 4) {         // all loads of four K-blocks first
                Frag8 a[4], b[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int c0 = (k0 + u) * 16 + 4 * g;
                    float2 x[4], y[4];
                    if (mat) grad_out4(row, c0, x);
                    else rec4(Frow, row, C, c0, x);
                    rec4(Drow, jcol, C, c0, y);                    // Delta^*: conj(Delta[jcol][cc])
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        a[u].v[2 * r] = x[r].x;
                        a[u].v[2 * r + 1] = x[r].y;
                        bpair(b[u], r, y[r].x, -y[r].y, qp);
                    }
                }
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (k0 + u < nkb) mma<P>(acc, a[u], b[u]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = rb * 16 + 4 * g + r;
                if (mat == 0) {
                    if (jcol < t) g2f[2 * (t * LDG + jcol) + qp] = -sm.beta[t] * acc[r];
                } else {
                    if (jcol <= t) g2f[2 * (jcol * LDG + t) + qp] = acc[r];
                }
            }
        }
    }
    __syncthreads();

    // ================================================================ G_Ki, G_Qg, G_Kg
    // Tile it of wave w covers channel block (w + 8 it) % 8 = w, so each wave collects the
    // dL/dg_C shares of its channel block in gsum.  The three products run one after another,
    // each holding only its own operands in registers.
    constexpr int PER = (NCT + GW - 1) / GW;
    f32x4 gki[PER], gqg[PER], gkg[PER];
    float gsum = 0.f;
    // left operand rows (K = value column): 0 conj(Delta), 1 G_R, 2 -G_E = -beta G_F
    auto left4 = [&](int kind, int row, int c0, Frag8& a) {
        float2 x[4];
        if (kind == 0) rec4(Drow, row, C, c0, x);
        else if (kind == 1) grad_out4(row, c0, x);
        else rec4(Frow, row, C, c0, x);
        const float sc = kind == 2 ? -sm.beta[min(row, C - 1)] : 1.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            a.v[2 * r] = sc * x[r].x;
            a.v[2 * r + 1] = kind == 0 ? -x[r].y : sc * x[r].y;
        }
    };
    // right operand (K = value column, output column icol): 0 G^T, 1 S^*
    auto right4 = [&](int kind, int icol, int c0, Frag8& b) {
        float2 y[4];
        rec4(kind == 0 ? Grec : Srec, icol, m, c0, y);
#pragma unroll
        for (int r = 0; r < 4; ++r) bpair(b, r, y[r].x, kind == 0 ? y[r].y : -y[r].y, qp);
    };
    // acc += (left kind lk) (right kind rk) over the value columns, two K-blocks of loads at a time
    auto value_product = [&](f32x4& acc, int lk, int rk, int row, int icol) {
        for (int k0 = 0; k0 < nkb; k0 += 2) {
            Frag8 a[2], b[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                left4(lk, row, (k0 + u) * 16 + 4 * g, a[u]);
                right4(rk, icol, (k0 + u) * 16 + 4 * g, b[u]);
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
                if (k0 + u < nkb) mma<P>(acc, a[u], b[u]);
        }
    };
    // a C x C operand fragment from g2: G_L' (strict lower at g2[t][j]) or G_A (lower, at g2[j][t])
    auto cc_frag = [&](bool transposed_store, int row, int kb, int lo, Frag8& a) {
        // lo: 0 -> jt < row, 1 -> jt <= row, 2 -> jt > row, 3 -> jt >= row
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int jt = kb * 16 + 4 * g + r;
            const bool ok = lo == 0 ? jt < row : lo == 1 ? jt <= row : lo == 2 ? jt > row : jt >= row;
            const float2 x = masked(ok, pin(transposed_store ? sm.g2[jt * LDG + row] : sm.g2[row * LDG + jt]));
            a.v[2 * r] = x.x;
            a.v[2 * r + 1] = x.y;
        }
    };
    auto lds_right = [&](const float2* X, int kb, int icol, Frag8& b) {   // conj(X[jt][icol])
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float2 y = X[(kb * 16 + 4 * g + r) * LDX + icol];
            bpair(b, r, y.x, -y.y, qp);
        }
    };
    // G_Ki = conj(Delta) G^T diag(conj(g_C)) + G_L'^T conj(conj(K)G) + G_A^T conj(conj(Q)G)
#pragma unroll
    for (int it = 0; it < PER; ++it) {
        const int tile = wave + GW * it;
        gki[it] = zero4();
        if (tile >= NCT) continue;
        const int rb = tile / (2 * MP / 16);
        const int icol = (tile - rb * (2 * MP / 16)) * 8 + (c >> 1);
        const int row = rb * 16 + c;
        value_product(gki[it], 0, 0, row, icol);
        // dL/dg_C, second part: column sums of G_Yp * conj(K/G)
        {
            float part = 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float2 kv = sm.ki[(rb * 16 + 4 * g + r) * LDX + icol];
                const float own = gki[it][r], oth = partner(own);
                part += qp ? (own * kv.x - oth * kv.y) : (own * kv.x + oth * kv.y);
            }
            part += __shfl_xor(part, 16);
            part += __shfl_xor(part, 32);
            gsum += part;
        }
        // G_Yp diag(conj(g_C))
        {
            const float2 gg = sm.gc[icol];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float own = gki[it][r], oth = partner(own);
                gki[it][r] = qp ? (gg.x * own - gg.y * oth) : (gg.x * own + gg.y * oth);
            }
        }
#pragma unroll
        for (int kb = rb; kb < NRB; ++kb) {
            Frag8 a, b;
            cc_frag(true, row, kb, 2, a);              // G_L'^T[row][jt] = G_L'[jt][row], jt > row
            lds_right(sm.kg, kb, icol, b);
            mma<P>(gki[it], a, b);
            cc_frag(false, row, kb, 3, a);             // G_A^T[row][jt] = G_A[jt][row], jt >= row
            lds_right(sm.qg, kb, icol, b);
            mma<P>(gki[it], a, b);
        }
    }
    // G_Qg = G_R S^* + G_A conj(K/G),  G_Kg = -G_E S^* + G_L' conj(K/G)
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
        for (int it = 0; it < PER; ++it) {
            const int tile = wave + GW * it;
            f32x4& acc = pass == 0 ? gqg[it] : gkg[it];
            acc = zero4();
            if (tile >= NCT) continue;
            const int rb = tile / (2 * MP / 16);
            const int icol = (tile - rb * (2 * MP / 16)) * 8 + (c >> 1);
            const int row = rb * 16 + c;
            value_product(acc, pass == 0 ? 1 : 2, 1, row, icol);
#pragma unroll
            for (int kb = 0; kb <= rb; ++kb) {
                Frag8 a, b;
                if (pass == 0) cc_frag(true, row, kb, 1, a);    // G_A[row][jt], jt <= row
                else cc_frag(false, row, kb, 0, a);             // G_L'[row][jt], jt < row
                lds_right(sm.ki, kb, icol, b);
                mma<P>(acc, a, b);
            }
        }
    }
    if (g == 0) {                                      // one owner lane per element of ggc
        const int icol = wave * 8 + (c >> 1);
        if (icol < m) ggc[2 * icol + qp] += gsum;
    }
    __syncthreads();                                   // every read of qg, kg, ki done
    {
        float* qgf = reinterpret_cast<float*>(sm.qg);
        float* kgf = reinterpret_cast<float*>(sm.kg);
        float* kif = reinterpret_cast<float*>(sm.ki);
#pragma unroll
        for (int it = 0; it < PER; ++it) {
            const int tile = wave + GW * it;
            if (tile >= NCT) continue;
            const int rb = tile / (2 * MP / 16);
            const int icol = (tile - rb * (2 * MP / 16)) * 8 + (c >> 1);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int e = 2 * ((rb * 16 + 4 * g + r) * LDX + icol) + qp;
                qgf[e] = gki[it][r];                   // G_Ki
                kgf[e] = gqg[it][r];                   // G_Qg
                kif[e] = gkg[it][r];                   // G_Kg
            }
        }
    }
    __syncthreads();

    // ================================================================ elementwise, suffix sums
    {
        const TIN* gq = static_cast<const TIN*>(args.q);
        const TIN* gk = static_cast<const TIN*>(args.k);
        const TIN* ga = static_cast<const TIN*>(args.alpha);
        TIN* dq = static_cast<TIN*>(A.dq);
        TIN* dk = static_cast<TIN*>(A.dk);
        TIN* dal = static_cast<TIN*>(A.dalpha);
        TIN* dth = static_cast<TIN*>(A.dtheta);
        const int i = tid & 63, seg = (tid >> 6) & 3;
        const bool worker = tid < NTHR;                // the load stage's thread mapping
        // g of this thread's tokens: running sums of log alpha and theta over its segment,
        // offset by the segments before it
        float2 gkeep[SEG];
        {
            const TIN* gth = static_cast<const TIN*>(args.theta);
            float la[SEG], ph[SEG];
            float sa = 0.f, sp2 = 0.f;
#pragma unroll
            for (int u = 0; u < SEG; ++u) {
                const int t = t0 + seg * SEG + u;
                const bool ok = t < T && i < m;
                const long e = base_tm + static_cast<long>(min(t, T - 1)) * m + min(i, m - 1);
                const float a_ld = pin(Elem<TIN>::load(ga, e));
                const float th = masked(ok, Elem<TIN>::load(gth, e));
                sa += __logf(ok ? a_ld : 1.f);
                sp2 += th;
                la[u] = sa;
                ph[u] = sp2;
            }
            if (worker) {
                sm.sega[seg][i] = sa;
                sm.segp[seg][i] = sp2;
            }
            __syncthreads();
            float oa = 0.f, op2 = 0.f;
            for (int s2 = 0; s2 < seg; ++s2) {
                oa += sm.sega[s2][i];
                op2 += sm.segp[s2][i];
            }
#pragma unroll
            for (int u = 0; u < SEG; ++u) {
                const float e = __expf(la[u] + oa);
                float sn, cs;
                __sincosf(ph[u] + op2, &sn, &cs);
                gkeep[u] = make_float2(e * cs, e * sn);
            }
            __syncthreads();                           // before sega / segp are reused below
        }
        float gl[SEG], gp[SEG];
        float sl = 0.f, sp = 0.f;
#pragma unroll
        for (int u = SEG - 1; u >= 0; --u) {
            if (!worker) break;
            const int tl = seg * SEG + u;
            const int t = t0 + tl;
            const bool ok = t < T && i < m;
            const long e = base_tm + static_cast<long>(min(t, T - 1)) * m + min(i, m - 1);
            const float2 qq = masked(ok, Elem<TIN>::load2(gq, e));
            const float2 kk = masked(ok, Elem<TIN>::load2(gk, e));
            const float2 gqv = sm.kg[tl * LDX + i], gkv = sm.ki[tl * LDX + i], gkiv = sm.qg[tl * LDX + i];
            const float2 gg = gkeep[u];
            const float inv2 = 1.f / (gg.x * gg.x + gg.y * gg.y);
            const float2 gi = make_float2(gg.x * inv2, -gg.y * inv2);            // 1 / g
            // dq = g conj(G_Qg); dk = g conj(G_Kg) + conj(1/g) G_Ki
            const float2 vq = make_float2(gg.x * gqv.x + gg.y * gqv.y, gg.y * gqv.x - gg.x * gqv.y);
            const float2 vk = make_float2(gg.x * gkv.x + gg.y * gkv.y + gi.x * gkiv.x + gi.y * gkiv.y,
                                          gg.y * gkv.x - gg.x * gkv.y + gi.x * gkiv.y - gi.y * gkiv.x);
            if (ok) {          // (a worker thread)
                Elem<TIN>::store2(dq, e, vq.x, vq.y);
                Elem<TIN>::store2(dk, e, vk.x, vk.y);
            }
            // dL/dg = q G_Qg + k G_Kg - conj(k / g^2) G_Ki
            const float2 kg2 = make_float2(kk.x * gi.x - kk.y * gi.y, kk.x * gi.y + kk.y * gi.x);     // k / g
            const float2 kg3 = make_float2(kg2.x * gi.x - kg2.y * gi.y, kg2.x * gi.y + kg2.y * gi.x); // k / g^2
            float2 dg = make_float2(qq.x * gqv.x - qq.y * gqv.y + kk.x * gkv.x - kk.y * gkv.y
                                        - (kg3.x * gkiv.x + kg3.y * gkiv.y),
                                    qq.x * gqv.y + qq.y * gqv.x + kk.x * gkv.y + kk.y * gkv.x
                                        - (kg3.x * gkiv.y - kg3.y * gkiv.x));
            if (tl == C - 1 && i < m) {
                dg.x += ggc[2 * i];
                dg.y += ggc[2 * i + 1];
            }
            // dL/dz = conj(g) dL/dg, suffix sums over the chunk
            sl += gg.x * dg.x + gg.y * dg.y;
            sp += gg.x * dg.y - gg.y * dg.x;
            gl[u] = sl;
            gp[u] = sp;
        }
        if (worker) {
            sm.sega[seg][i] = sl;
            sm.segp[seg][i] = sp;
        }
        __syncthreads();
        if (!worker) return;
        float ol = 0.f, op = 0.f;
        for (int s2 = seg + 1; s2 < 4; ++s2) {
            ol += sm.sega[s2][i];
            op += sm.segp[s2][i];
        }
#pragma unroll
        for (int u = 0; u < SEG; ++u) {
            const int t = t0 + seg * SEG + u;
            if (t < T && i < m) {
                const long e = base_tm + static_cast<long>(t) * m + i;
                Elem<TIN>::store(dal, e, (gl[u] + ol) / Elem<TIN>::load(ga, e));
                Elem<TIN>::store(dth, e, gp[u] + op);
            }
        }
        if (tid < C && t0 + tid < T) {
            float db = 0.f;
#pragma unroll
            for (int w = 0; w < GW; ++w) db += dbeta_part[w][tid];
            Elem<TIN>::store(static_cast<TIN*>(A.dbeta), bh * static_cast<long>(T) + t0 + tid, db);
        }
    }
}

template <int P, typename TIN, typename TOUT>
static hipError_t launch_grad_t(const GradLaunch& L, hipStream_t st)
{
    GradArgs a{};
    a.in.q = L.q; a.in.k = L.k; a.in.v = L.v; a.in.alpha = L.alpha; a.in.theta = L.theta;
    a.in.beta = L.beta;
    a.in.T = L.T; a.in.m = L.m; a.in.n = L.n;
    a.in.amin = 0.f; a.in.aspan = 1.f; a.in.tmax = 0.f; a.in.eps = 0.f;
    a.dO = L.dO;
    a.S_rec = L.S_rec; a.G_rec = L.G_rec; a.D_rows = L.D_rows; a.F_rows = L.F_rows;
    a.dq = L.dq; a.dk = L.dk; a.dalpha = L.dalpha; a.dtheta = L.dtheta; a.dbeta = L.dbeta;
    const long nchunks = (L.T + L.C - 1) / L.C;
    const dim3 grid(static_cast<unsigned>(static_cast<long>(L.B) * L.H * nchunks));
    switch (L.C) {
        case 16: hipLaunchKernelGGL((grad_kernel<P, TIN, TOUT, 16>), grid, dim3(GW * 64), 0, st, a); break;
        case 32: hipLaunchKernelGGL((grad_kernel<P, TIN, TOUT, 32>), grid, dim3(GW * 64), 0, st, a); break;
        case 64: hipLaunchKernelGGL((grad_kernel<P, TIN, TOUT, 64>), grid, dim3(GW * 64), 0, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_chunk_grad(const GradLaunch& L, hipStream_t st)
{
    // bf16 inputs take bf16 matrix-core operands (fp32 accumulation and records)
    if (L.in_bf16)
        return L.out_bf16 ? launch_grad_t<PREC_BF16, uint16_t, uint16_t>(L, st)
                          : launch_grad_t<PREC_BF16, uint16_t, float>(L, st);
    return L.out_bf16 ? launch_grad_t<PREC_F32, float, uint16_t>(L, st) : launch_grad_t<PREC_F32, float, float>(L, st);
}

}  // namespace sfda
