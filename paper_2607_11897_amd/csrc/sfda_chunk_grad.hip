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
// Products over the value dimension take their operands from LDS: the records are staged
// a block of value columns at a time (every load of a block in flight together) and each
// product accumulates over the blocks in registers, so the pass waits on global memory
// once per block instead of once per product; products over tokens read the decay-scaled
// operands from LDS.  The C x C gradients G_L' and G_A share one LDS block (G_L' strict
// lower, G_A^T upper with the diagonal).  The library launches it at C = 16 (the chunk length
// of the whole backward).
#include <type_traits>

#include "sfda_chunk_common.h"

namespace sfda {

constexpr int GW = 8;        // waves per workgroup

struct GradArgs {
    ChunkArgs in;                          // q, k, v, alpha, theta, beta, T, m, n
    const void* dO;
    const float *S_rec, *G_rec, *D_rows, *F_rows;
    void *dq, *dk, *dalpha, *dtheta, *dbeta;
};

// ---------------------------------------------------------------- staged record blocks
// The products over the value dimension read a block of NB value columns of S, G (state
// rows x NB) and of Delta, G_F, G_R (tokens x NB) from LDS, staged once per block with every
// load of the block in flight together.  The bf16 path keeps them as bf16 pairs (its matrix
// cores round the operands to bf16 anyway; the fp32 records stay the source of the
// elementwise sums), the fp32 path as fp32.  Rows are 272 bytes: a 16-byte fragment read by
// 16 lanes of different rows touches every bank once.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

struct FragW { u32x4 w; };   // a lane's 8 bf16 operand values as 4 packed pairs

template <int P> struct Rec;

template <> struct Rec<PREC_BF16> {
    using E = uint32_t;      // (re, im) bf16 pair, re in the low half
    using Op = FragW;
    static constexpr int NB = 64, LD = 68;
    static __device__ __forceinline__ E pack(float2 x) {
        const f32x2 v = {x.x, x.y};
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
    }
    static __device__ __forceinline__ float re(E w) { return __uint_as_float(w << 16); }
    static __device__ __forceinline__ float im(E w) { return __uint_as_float(w & 0xFFFF0000u); }
    // the B pair of bpair for y (cj: for conj(y)) and output column part q, on the packed
    // word: part 1 swaps the halves (a byte permute), the sign flips are one xor
    static __device__ __forceinline__ uint32_t bword(E w, bool cj, int q) {
        const uint32_t sel = q ? 0x01000302u : 0x03020100u;
        const uint32_t flip = q ? (cj ? 0x8000u : 0u) : (cj ? 0u : 0x80000000u);
        return __builtin_amdgcn_perm(w, w, sel) ^ flip;
    }
    // A fragment: four consecutive entries of one row (16-byte aligned), cj conjugates
    static __device__ __forceinline__ Op left(const E* p, bool cj) {
        u32x4 x = *reinterpret_cast<const u32x4*>(p);
        if (cj) x ^= 0x80000000u;
        return Op{x};
    }
    static __device__ __forceinline__ Op right(E y0, E y1, E y2, E y3, bool cj, int q) {
        const u32x4 x = {bword(y0, cj, q), bword(y1, cj, q), bword(y2, cj, q), bword(y3, cj, q)};
        return Op{x};
    }
    static __device__ __forceinline__ Op right4(const E* p, bool cj, int q) {
        const u32x4 x = *reinterpret_cast<const u32x4*>(p);
        return right(x[0], x[1], x[2], x[3], cj, q);
    }
    static __device__ __forceinline__ Op conv(const Frag8& f) {
        u32x4 x;
#pragma unroll
        for (int r = 0; r < 4; ++r) x[r] = pack(make_float2(f.v[2 * r], f.v[2 * r + 1]));
        return Op{x};
    }
    static __device__ __forceinline__ void mma(f32x4& acc, const Op& a, const Op& b) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a.w),
                                                       __builtin_bit_cast(bf16x8, b.w), acc, 0, 0, 0);
    }
};

template <> struct Rec<PREC_F32> {
    using E = float2;
    using Op = Frag8;
    static constexpr int NB = 32, LD = 34;
    static __device__ __forceinline__ E pack(float2 x) { return x; }
    static __device__ __forceinline__ float re(E w) { return w.x; }
    static __device__ __forceinline__ float im(E w) { return w.y; }
    static __device__ __forceinline__ Op left(const E* p, bool cj) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        const float4 b = *reinterpret_cast<const float4*>(p + 2);
        const float s = cj ? -1.f : 1.f;
        Op f;
        f.v[0] = a.x; f.v[1] = s * a.y; f.v[2] = a.z; f.v[3] = s * a.w;
        f.v[4] = b.x; f.v[5] = s * b.y; f.v[6] = b.z; f.v[7] = s * b.w;
        return f;
    }
    static __device__ __forceinline__ Op right(E y0, E y1, E y2, E y3, bool cj, int q) {
        const float s = cj ? -1.f : 1.f;
        Op f;
        bpair(f, 0, y0.x, s * y0.y, q);
        bpair(f, 1, y1.x, s * y1.y, q);
        bpair(f, 2, y2.x, s * y2.y, q);
        bpair(f, 3, y3.x, s * y3.y, q);
        return f;
    }
    static __device__ __forceinline__ Op right4(const E* p, bool cj, int q) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        const float4 b = *reinterpret_cast<const float4*>(p + 2);
        return right(make_float2(a.x, a.y), make_float2(a.z, a.w), make_float2(b.x, b.y),
                     make_float2(b.z, b.w), cj, q);
    }
    static __device__ __forceinline__ Op conv(const Frag8& f) { return f; }
    static __device__ __forceinline__ void mma(f32x4& acc, const Op& a, const Op& b) {
        sfda::mma<PREC_F32>(acc, a, b);
    }
};

template <int P, int C>
struct GradSmem {
    using E = typename Rec<P>::E;
    static constexpr int LD = Rec<P>::LD;
    ChunkSmem<C> ch;
    alignas(16) E S[MP * LD];          // state entering the chunk
    alignas(16) E G[MP * LD];          // dL/dS of the state leaving it
    alignas(16) E D[C * LD];           // Delta
    alignas(16) E F[C * LD];           // G_F
    alignas(16) E R[C * LD];           // G_R = conj(dL/do)
    float dbeta_part[GW][C];           // per-wave shares of dbeta
    float ggc[2 * MP];                 // dL/dg_C (complex)
};

template <int P, typename TIN, typename TOUT, int C>
__global__ __launch_bounds__(GW * 64, C <= 16 ? 4 : 2) void grad_kernel(GradArgs A)
{
    using RC = Rec<P>;
    using Op = typename RC::Op;
    constexpr int NB = RC::NB, LD = RC::LD;
    constexpr int NRB = C / 16;
    constexpr int SEG = C / 4;
    constexpr int LDG = ChunkSmem<C>::LDG;
    constexpr int NCT = NRB * (2 * MP / 16);        // C x m output tiles (16 tokens x 8 channels)
    constexpr int NT1 = NRB * (NRB + 1);            // causal tiles of a C x C matrix
    constexpr int PER = (NCT + GW - 1) / GW;        // C x m tiles per wave
    constexpr int NGA = (2 * NT1 + GW - 1) / GW;    // G_A / G_L' tiles per wave
    constexpr int RPI = GW * 64 / NB;               // record rows per staging step
    constexpr int NS = MP / RPI;                    // staged S, G entries per thread
    constexpr int NR = C / RPI;                     // staged Delta, G_F, G_R entries per thread
    static_assert(NR >= 1 && NB % 16 == 0 && NB / 8 <= GW, "staging shape");
    __shared__ GradSmem<P, C> gs;
    ChunkSmem<C>& sm = gs.ch;
#ifdef SFDA_LDS_POISON
    // every LDS entry this workgroup reads is written by it first
    lds_poison(&gs, sizeof(gs), threadIdx.x, GW * 64);
    __syncthreads();
#endif

    const ChunkArgs& args = A.in;
    const int T = args.T, m = args.m, n = args.n;
    const int nchunks = (T + C - 1) / C;
    const long bh = blockIdx.x / nchunks;
    const int ch = static_cast<int>(blockIdx.x - bh * nchunks);
    const int t0 = ch * C;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int c = lane & 15, g = lane >> 4, qp = lane & 1;

    const float2* Srec = reinterpret_cast<const float2*>(A.S_rec) + (bh * nchunks + ch) * static_cast<long>(m) * n;
    const float2* Grec = reinterpret_cast<const float2*>(A.G_rec) + (bh * nchunks + ch) * static_cast<long>(m) * n;
    const float2* Drow = reinterpret_cast<const float2*>(A.D_rows) + (bh * nchunks * static_cast<long>(C) + t0) * n;
    const float2* Frow = reinterpret_cast<const float2*>(A.F_rows) + (bh * nchunks * static_cast<long>(C) + t0) * n;
    const TOUT* gdO = static_cast<const TOUT*>(A.dO);
    const TIN* gv = static_cast<const TIN*>(args.v);
    const long base_tn = bh * static_cast<long>(T) * n;
    const long base_tm = bh * static_cast<long>(T) * m;

    // ------------------------------------------------------------ staging
    // thread tid covers column tid % NB of rows tid / NB + RPI u (consecutive lanes read
    // consecutive columns); the H stage's conj(V) parts go straight to registers
    struct Raw {
        float2 s[NS], g[NS], d[NR], f[NR], r[NR];
        typename RC::E v[NRB][4];                   // raw v entries (parts taken in the H stage)
    };
    const int scol = tid % NB, srow = tid / NB;
    const int rows_in = min(C, T - t0);             // tokens of this chunk inside the sequence
    const rsrc_t rS = buf(Srec, static_cast<long>(m) * n * 8), rG = buf(Grec, static_cast<long>(m) * n * 8);
    const rsrc_t rD = buf(Drow, static_cast<long>(C) * n * 8), rF = buf(Frow, static_cast<long>(C) * n * 8);
    const rsrc_t rO = buf(gdO + 2 * (base_tn + static_cast<long>(t0) * n), static_cast<long>(rows_in) * n * 2 * sizeof(TOUT));
    const rsrc_t rV = buf(gv + 2 * (base_tn + static_cast<long>(t0) * n), static_cast<long>(rows_in) * n * 2 * sizeof(TIN));
    auto fetch = [&](int n0, Raw& x) {
        const int j = n0 + scol;
        const bool jok = j < n;
#pragma unroll
        for (int u = 0; u < NS; ++u) {              // rows past m lie past the resource
            const uint32_t off = jok ? static_cast<uint32_t>(((srow + RPI * u) * n + j) * 8) : OOR;
            x.s[u] = ld_c64(rS, off);
            x.g[u] = ld_c64(rG, off);
        }
#pragma unroll
        for (int u = 0; u < NR; ++u) {              // tokens past T lie past rO
            const uint32_t e = static_cast<uint32_t>((srow + RPI * u) * n + j);
            x.d[u] = ld_c64(rD, jok ? e * 8 : OOR);
            x.f[u] = ld_c64(rF, jok ? e * 8 : OOR);
            x.r[u] = ld_cplx<TOUT>(rO, jok ? e * 2 * static_cast<uint32_t>(sizeof(TOUT)) : OOR);
        }
        const int jv = n0 + wave * 8 + (c >> 1);
        const bool vok = wave < NB / 8 && jv < n;
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t e = static_cast<uint32_t>((rb * 16 + 4 * g + r) * n + jv);
                const uint32_t off = vok ? e * 2 * static_cast<uint32_t>(sizeof(TIN)) : OOR;
                if constexpr (sizeof(TIN) == 2) {          // a complex bf16 pair
                    const uint32_t w = __builtin_amdgcn_raw_buffer_load_b32(rV, off, 0, 0);
                    if constexpr (P == PREC_BF16) x.v[rb][r] = w;
                    else x.v[rb][r] = make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
                } else {
                    x.v[rb][r] = ld_c64(rV, off);
                }
            }
    };
    // put also adds the block's share of dL/dg_C's first part, rowsum(G * conj(S)) from the
    // fp32 records (one row per NB lanes; lane scol == 0 owns the row's entry of ggc)
    auto put = [&](const Raw& x, bool first) {
#pragma unroll
        for (int u = 0; u < NS; ++u) {
            const int i = srow + RPI * u;
            gs.S[i * LD + scol] = RC::pack(x.s[u]);
            gs.G[i * LD + scol] = RC::pack(x.g[u]);
            float px = x.g[u].x * x.s[u].x + x.g[u].y * x.s[u].y;
            float py = x.g[u].y * x.s[u].x - x.g[u].x * x.s[u].y;
#pragma unroll
            for (int sh = 1; sh < NB; sh <<= 1) {
                px += __shfl_xor(px, sh);
                py += __shfl_xor(py, sh);
            }
            if (scol == 0) {
                gs.ggc[2 * i] = first ? px : gs.ggc[2 * i] + px;
                gs.ggc[2 * i + 1] = first ? py : gs.ggc[2 * i + 1] + py;
            }
        }
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int tl = srow + RPI * u;
            gs.D[tl * LD + scol] = RC::pack(x.d[u]);
            gs.F[tl * LD + scol] = RC::pack(x.f[u]);
            gs.R[tl * LD + scol] = RC::pack(make_float2(x.r[u].x, -x.r[u].y));
        }
    };

    // ------------------------------------------------------------ load stage, L'
    // (the load stage and the elementwise stage work on the first 256 threads; the latter
    // forms g again rather than holding it in registers through the whole kernel)
    Raw raw;
    {
        // the first record block, then alpha, theta, beta, then q, k
        fetch(0, raw);
        InPre<C> pf;
        prefetch_inputs<TIN, C, true>(args, bh, t0, tid, pf);
        float2 gkeep[SEG];
        stage_load<TIN, C, false, false, false, ChunkSmem<C>, true, true>(sm, args, bh, t0, tid, gkeep, &pf);
    }
    put(raw, true);
    __syncthreads();
    stage_gram<P, C, false, false, ChunkSmem<C>, GW>(sm, tid);   // L'
    __syncthreads();

    // ------------------------------------------------------------ value-column blocks
    float dacc[NRB][4];
    f32x4 gacc[NGA], gki[PER], gqg[PER], gkg[PER];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 4; ++r) dacc[rb][r] = 0.f;
#pragma unroll
    for (int s = 0; s < NGA; ++s) gacc[s] = zero4();
#pragma unroll
    for (int it = 0; it < PER; ++it) {
        gki[it] = zero4();
        gqg[it] = zero4();
        gkg[it] = zero4();
    }
    // causal C x C tile -> (matrix, row block, column block)
    auto ga_tile = [&](int tile, int& mat, int& rb, int& cb) {
        mat = tile / NT1;
        int rem = tile - mat * NT1;
        rb = 0;
        while (rem >= min(C / 8, 2 * rb + 2)) { rem -= min(C / 8, 2 * rb + 2); ++rb; }
        cb = rem;
    };
    const int nblk = (n + NB - 1) / NB;
    for (int blk = 0; blk < nblk; ++blk) {
        if (blk > 0) {
            __syncthreads();                           // every read of the previous block done
            fetch(blk * NB, raw);
            put(raw, false);
            __syncthreads();
        }
        // H = E - L' Delta and the dbeta shares (Re conj(G_F) H), column block `wave`; each
        // wave sums in registers, the per-wave shares are added in a fixed order at the end
        if (wave < NB / 8) {
            const int jl = wave * 8 + (c >> 1);
            Op sbf[MP / 16], dbf[NRB];
#pragma unroll
            for (int kb = 0; kb < MP / 16; ++kb) {
                const int i0 = kb * 16 + 4 * g;
                sbf[kb] = RC::right(gs.S[i0 * LD + jl], gs.S[(i0 + 1) * LD + jl], gs.S[(i0 + 2) * LD + jl],
                                    gs.S[(i0 + 3) * LD + jl], false, qp);
            }
#pragma unroll
            for (int kb = 0; kb < NRB; ++kb) {
                const int i0 = kb * 16 + 4 * g;
                dbf[kb] = RC::right(gs.D[i0 * LD + jl], gs.D[(i0 + 1) * LD + jl], gs.D[(i0 + 2) * LD + jl],
                                    gs.D[(i0 + 3) * LD + jl], false, qp);
            }
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb) {
                const int row = rb * 16 + c;
                f32x4 pw = zero4();                    // (conj(K) G) S + L' Delta
#pragma unroll
                for (int kb = 0; kb < MP / 16; ++kb) {
                    Frag8 a;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float2 x = sm.kg[row * LDX + kb * 16 + 4 * g + r];
                        a.v[2 * r] = x.x;
                        a.v[2 * r + 1] = x.y;
                    }
                    RC::mma(pw, RC::conv(a), sbf[kb]);
                }
#pragma unroll
                for (int kb = 0; kb <= rb; ++kb) {
                    Frag8 a;
                    float2 xs[4];
                    lds_masked4([&](int r) { return sm.g2[row * LDG + kb * 16 + 4 * g + r]; },
                                [&](int r) { return kb * 16 + 4 * g + r < row; }, xs);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        a.v[2 * r] = xs[r].x;
                        a.v[2 * r + 1] = xs[r].y;
                    }
                    RC::mma(pw, RC::conv(a), dbf[kb]);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const auto f = gs.F[(rb * 16 + 4 * g + r) * LD + jl];
                    const auto vw = raw.v[rb][r];
                    const float h = (qp ? -RC::im(vw) : RC::re(vw)) - pw[r];   // H, this lane's part
                    float prod = (qp ? RC::im(f) : RC::re(f)) * h;  // Re(conj(G_F) H) share
                    prod += __shfl_xor(prod, 1);
                    prod += __shfl_xor(prod, 2);
                    prod += __shfl_xor(prod, 4);
                    prod += __shfl_xor(prod, 8);
                    dacc[rb][r] += prod;
                }
            }
        }
        // G_A = tril(G_R Delta^*) and G_F Delta^* (G_L' after the loop), over this block
#pragma unroll
        for (int s = 0; s < NGA; ++s) {
            const int tile = wave + GW * s;
            if (tile >= 2 * NT1) continue;
            int mat, rb, cb;
            ga_tile(tile, mat, rb, cb);
            const int row = rb * 16 + c;
            const int jcol = cb * 8 + (c >> 1);
#pragma unroll
            for (int kb = 0; kb < NB / 16; ++kb) {
                const int c0 = kb * 16 + 4 * g;
                const Op a = RC::left(mat ? &gs.R[row * LD + c0] : &gs.F[row * LD + c0], false);
                RC::mma(gacc[s], a, RC::right4(&gs.D[jcol * LD + c0], true, qp));
            }
        }
        // value-column parts of G_Ki (conj(Delta) G^T), G_Qg (G_R S^*) and G_F S^*
#pragma unroll
        for (int it = 0; it < PER; ++it) {
            const int tile = wave + GW * it;
            if (tile >= NCT) continue;
            const int rb = tile / (2 * MP / 16);
            const int icol = (tile - rb * (2 * MP / 16)) * 8 + (c >> 1);
            const int row = rb * 16 + c;
#pragma unroll
            for (int kb = 0; kb < NB / 16; ++kb) {
                const int c0 = kb * 16 + 4 * g;
                RC::mma(gki[it], RC::left(&gs.D[row * LD + c0], true), RC::right4(&gs.G[icol * LD + c0], false, qp));
                const Op bs = RC::right4(&gs.S[icol * LD + c0], true, qp);
                RC::mma(gqg[it], RC::left(&gs.R[row * LD + c0], false), bs);
                RC::mma(gkg[it], RC::left(&gs.F[row * LD + c0], false), bs);
            }
        }
    }
    __syncthreads();                                   // every read of L' and of the records done

    // ------------------------------------------------------------ C x C gradients, dL/dg_C
    if (c == 0) {
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
            for (int r = 0; r < 4; ++r) gs.dbeta_part[wave][rb * 16 + 4 * g + r] = dacc[rb][r];
    }
    // G_L' = D_beta strict_tril(-G_F Delta^*) at g2[t][j], G_A^T (upper with the diagonal)
    {
        float* g2f = reinterpret_cast<float*>(sm.g2);
#pragma unroll
        for (int s = 0; s < NGA; ++s) {
            const int tile = wave + GW * s;
            if (tile >= 2 * NT1) continue;
            int mat, rb, cb;
            ga_tile(tile, mat, rb, cb);
            const int jcol = cb * 8 + (c >> 1);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = rb * 16 + 4 * g + r;
                if (mat == 0) {
                    if (jcol < t) g2f[2 * (t * LDG + jcol) + qp] = -sm.beta[t] * gacc[s][r];
                } else {
                    if (jcol <= t) g2f[2 * (jcol * LDG + t) + qp] = gacc[s][r];
                }
            }
        }
    }
    __syncthreads();

    // ------------------------------------------------------------ G_Ki, G_Qg, G_Kg
    // Tile it of wave w covers channel block (w + 8 it) % 8 = w, so each wave collects the
    // dL/dg_C shares of its channel block in gsum.
    float gsum = 0.f;
    // a C x C operand fragment from g2: G_L' (strict lower at g2[t][j]) or G_A (lower, at g2[j][t])
    auto cc_frag = [&](bool transposed_store, int row, int kb, int lo) {
        // lo: 0 -> jt < row, 1 -> jt <= row, 2 -> jt > row, 3 -> jt >= row
        Frag8 a;
        float2 xs[4];
        lds_masked4([&](int r) {
                        const int jt = kb * 16 + 4 * g + r;
                        return transposed_store ? sm.g2[jt * LDG + row] : sm.g2[row * LDG + jt];
                    },
                    [&](int r) {
                        const int jt = kb * 16 + 4 * g + r;
                        return lo == 0 ? jt < row : lo == 1 ? jt <= row : lo == 2 ? jt > row : jt >= row;
                    }, xs);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            a.v[2 * r] = xs[r].x;
            a.v[2 * r + 1] = xs[r].y;
        }
        return RC::conv(a);
    };
    auto lds_right = [&](const float2* X, int kb, int icol) {   // conj(X[jt][icol])
        Frag8 b;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float2 y = X[(kb * 16 + 4 * g + r) * LDX + icol];
            bpair(b, r, y.x, -y.y, qp);
        }
        return RC::conv(b);
    };
#pragma unroll
    for (int it = 0; it < PER; ++it) {
        const int tile = wave + GW * it;
        if (tile >= NCT) continue;
        const int rb = tile / (2 * MP / 16);
        const int icol = (tile - rb * (2 * MP / 16)) * 8 + (c >> 1);
        const int row = rb * 16 + c;
        // dL/dg_C, second part: column sums of G_Yp * conj(K/G) (G_Yp = conj(Delta) G^T)
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
        // G_Kg's value part is -G_E S^* = -D_beta (G_F S^*)
#pragma unroll
        for (int r = 0; r < 4; ++r) gkg[it][r] *= -sm.beta[rb * 16 + 4 * g + r];
        // + G_L'^T conj(conj(K)G) + G_A^T conj(conj(Q)G); G_A's diagonal is left out of this
        // product and of G_Qg's (added in the elementwise stage, below)
#pragma unroll
        for (int kb = rb; kb < NRB; ++kb) {
            RC::mma(gki[it], cc_frag(true, row, kb, 2), lds_right(sm.kg, kb, icol));    // G_L'[jt][row], jt > row
            RC::mma(gki[it], cc_frag(false, row, kb, 2), lds_right(sm.qg, kb, icol));   // G_A[jt][row], jt > row
        }
        // G_Qg += G_A conj(K/G),  G_Kg += G_L' conj(K/G)
#pragma unroll
        for (int kb = 0; kb <= rb; ++kb) {
            const Op b = lds_right(sm.ki, kb, icol);
            RC::mma(gqg[it], cc_frag(true, row, kb, 0), b);                             // G_A[row][jt], jt < row
            RC::mma(gkg[it], cc_frag(false, row, kb, 0), b);                            // G_L'[row][jt], jt < row
        }
    }
    if (g == 0) {                                      // one owner lane per element of ggc
        const int icol = wave * 8 + (c >> 1);
        if (icol < m) gs.ggc[2 * icol + qp] += gsum;
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

    // ------------------------------------------------------------ elementwise, suffix sums
    {
        const TIN* gq = static_cast<const TIN*>(args.q);
        const TIN* gk = static_cast<const TIN*>(args.k);
        const TIN* ga = static_cast<const TIN*>(args.alpha);
        const TIN* gth = static_cast<const TIN*>(args.theta);
        TIN* dq = static_cast<TIN*>(A.dq);
        TIN* dk = static_cast<TIN*>(A.dk);
        TIN* dal = static_cast<TIN*>(A.dalpha);
        TIN* dth = static_cast<TIN*>(A.dtheta);
        const int i = tid & 63, seg = (tid >> 6) & 3;
        const bool worker = tid < NTHR;                // the load stage's thread mapping
        // every load of the stage at once: alpha, theta, q, k of this thread's tokens (zero
        // past T and past m)
        float av[SEG], la[SEG], ph[SEG];
        float2 qq[SEG], kk[SEG];
        {
            const long e0 = base_tm + static_cast<long>(t0) * m;
            const long bytes = static_cast<long>(rows_in) * m * sizeof(TIN);
            const rsrc_t ra = buf(ga + e0, bytes), rt = buf(gth + e0, bytes);
            const rsrc_t rq = buf(gq + 2 * e0, 2 * bytes), rk = buf(gk + 2 * e0, 2 * bytes);
#pragma unroll
            for (int u = 0; u < SEG; ++u) {
                const uint32_t e = static_cast<uint32_t>((seg * SEG + u) * m + i);
                const uint32_t o1 = i < m ? e * static_cast<uint32_t>(sizeof(TIN)) : OOR;
                const uint32_t o2 = i < m ? 2 * e * static_cast<uint32_t>(sizeof(TIN)) : OOR;
                av[u] = ld_real<TIN>(ra, o1);
                ph[u] = ld_real<TIN>(rt, o1);
                qq[u] = ld_cplx<TIN>(rq, o2);
                kk[u] = ld_cplx<TIN>(rk, o2);
            }
        }
        // g of this thread's tokens: running sums of log alpha and theta over its segment,
        // offset by the segments before it (padding is the identity token: alpha read as 0
        // there counts as 1); 1 / g from the negated sums (finite while the chunk's decay so
        // far is at least 2^-126, NaN past that, as in the load stage)
        float2 gkeep[SEG], gikeep[SEG];
        {
            float sa = 0.f, sp2 = 0.f;
#pragma unroll
            for (int u = 0; u < SEG; ++u) {
                const bool ok = t0 + seg * SEG + u < T && i < m;
                sa += __logf(av[u] + (ok ? 0.f : 1.f));
                sp2 = __builtin_amdgcn_fractf(__builtin_fmaf(ph[u], 0.15915494309189535f, sp2));   // revolutions
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
                const float A = la[u] + oa;
                const float e = __expf(A);
                const float ei = A >= -87.3365447f ? __expf(-A) : __builtin_nanf("");
                const float sn = __builtin_amdgcn_sinf(ph[u] + op2), cs = __builtin_amdgcn_cosf(ph[u] + op2);
                gkeep[u] = make_float2(e * cs, e * sn);
                gikeep[u] = make_float2(ei * cs, -ei * sn);
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
            const float2 gqv = sm.kg[tl * LDX + i], gkv = sm.ki[tl * LDX + i], gkiv = sm.qg[tl * LDX + i];
            const float2 gg = gkeep[u], gi = gikeep[u];                          // g, 1 / g
            const float2 q1 = qq[u], k1 = kk[u];
            const float2 kg2 = make_float2(k1.x * gi.x - k1.y * gi.y, k1.x * gi.y + k1.y * gi.x);     // k / g
            // G_A's diagonal a = G_A[t][t]: its terms in G_Qg and G_Ki, a conj(k / g) and
            // a q conj(g), go into dq and dk here in float32.  In dL/dz they cancel exactly
            // (A[t][t] = q_t . conj(k_t) does not depend on the decay), so dL/dz leaves both
            // out rather than subtracting two separately rounded products.
            const float2 ga = sm.g2[tl * LDG + tl];
            const float2 qcg = make_float2(q1.x * gg.x + q1.y * gg.y, q1.y * gg.x - q1.x * gg.y);    // q conj(g)
            const float2 gqf = make_float2(gqv.x + ga.x * kg2.x + ga.y * kg2.y, gqv.y + ga.y * kg2.x - ga.x * kg2.y);
            const float2 gkif = make_float2(gkiv.x + ga.x * qcg.x - ga.y * qcg.y, gkiv.y + ga.x * qcg.y + ga.y * qcg.x);
            // dq = g conj(G_Qg); dk = g conj(G_Kg) + conj(1/g) G_Ki
            const float2 vq = make_float2(gg.x * gqf.x + gg.y * gqf.y, gg.y * gqf.x - gg.x * gqf.y);
            const float2 vk = make_float2(gg.x * gkv.x + gg.y * gkv.y + gi.x * gkif.x + gi.y * gkif.y,
                                          gg.y * gkv.x - gg.x * gkv.y + gi.x * gkif.y - gi.y * gkif.x);
            if (ok) {          // (a worker thread)
                Elem<TIN>::store2(dq, e, vq.x, vq.y);
                Elem<TIN>::store2(dk, e, vk.x, vk.y);
            }
            // dL/dg = q G_Qg + k G_Kg - conj(k / g^2) G_Ki (+ dL/dg_C at the chunk's last
            // token), and dL/dz = conj(g) dL/dg: the last term becomes conj(k / g) G_Ki, so
            // no operand goes below 1 / g
            float2 dp = make_float2(q1.x * gqv.x - q1.y * gqv.y + k1.x * gkv.x - k1.y * gkv.y,
                                    q1.x * gqv.y + q1.y * gqv.x + k1.x * gkv.y + k1.y * gkv.x);
            if (tl == C - 1 && i < m) {
                dp.x += gs.ggc[2 * i];
                dp.y += gs.ggc[2 * i + 1];
            }
            // suffix sums of dL/dz over the chunk
            sl += gg.x * dp.x + gg.y * dp.y - (kg2.x * gkiv.x + kg2.y * gkiv.y);
            sp += gg.x * dp.y - gg.y * dp.x - (kg2.x * gkiv.y - kg2.y * gkiv.x);
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
                Elem<TIN>::store(dal, e, (gl[u] + ol) / av[u]);
                Elem<TIN>::store(dth, e, gp[u] + op);
            }
        }
        if (tid < C && t0 + tid < T) {
            float db = 0.f;
#pragma unroll
            for (int w = 0; w < GW; ++w) db += gs.dbeta_part[w][tid];
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
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_chunk_grad(const GradLaunch& L, hipStream_t st)
{
    // bf16 inputs take bf16 matrix-core operands (fp32 accumulation and records)
    if (bf16_operands(L.in_bf16, L.m))
        return L.out_bf16 ? launch_grad_t<PREC_BF16, uint16_t, uint16_t>(L, st)
                          : launch_grad_t<PREC_BF16, uint16_t, float>(L, st);
    if (L.in_bf16)          // a few key channels: fp32 operands
        return L.out_bf16 ? launch_grad_t<PREC_F32, uint16_t, uint16_t>(L, st)
                          : launch_grad_t<PREC_F32, uint16_t, float>(L, st);
    return L.out_bf16 ? launch_grad_t<PREC_F32, float, uint16_t>(L, st) : launch_grad_t<PREC_F32, float, float>(L, st);
}

}  // namespace sfda
