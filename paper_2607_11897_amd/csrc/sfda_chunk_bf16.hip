// Chunkwise SFDA forward for bfloat16 inputs on gfx950: a producer/consumer pipeline inside
// one workgroup per (batch, head, slice of value columns).
//
// Method.  The recurrence S_t = Lambda_t S_{t-1} + k_t delta_t with
// delta_t = beta_t (v_t^* - k_t^* Lambda_t S_{t-1}) is evaluated on blocks of 16 tokens.  For
// one block with entering state S, and g_t the product of lambda over the block's tokens up
// to t (the diagonal of the block's Gamma_t), unrolling it gives the chunk-WY factors of
// Thm 4.2 / Cor. 4.3 in closed form:
//   (I + D_beta L) Delta = D_beta (conj(V) - (conj(K) * G) S)          L[t, j] = k_t^* diag(g_t / g_j) k_j, j < t
//   O^*   = (conj(Q) * G) S + tril(A) Delta                             A[r, j] = q_r^* diag(g_r / g_j) k_j, j <= r
//   S_out = diag(g_16) S + (K * (g_16 / G))^T Delta
// -- the exact affine block transfer of Thm 4.4 (the paper's M is (I + L D_beta)^{-1}) with the
// prefix outputs of Thm 4.5.  The blocks are chained by the boundary-state scan (apply-transfer
// equation, Thm 6.1); a pipeline step takes four blocks (64 tokens).
//
// Decay range.  Every decay factor is a product of alphas over tokens inside one block,
// taken forwards from the block's start (P_t, in conj(Q) * G and conj(K) * G) or backwards
// from its end (Q_t, in K * (g_16 / G)), so these operands never exceed |q| or |k| and an
// underflow only ever drops a contribution that is itself below the float range.  Only the
// right operand of the block's own Gram matrices divides, k_j / P_j, and stays finite while
// the product of alpha over the block is at least 2^-126 (every alpha >= 0.0043 suffices);
// a step holding a block outside that range returns NaN from there on (its state is set to
// NaN).  Phases are kept as running sums of theta / 2 pi reduced to [0, 1) revolutions
// from the start of the sequence (a global frame: the state is held rotated by
// exp(-i phi) of the phase reached so far, and rotated back once at the end), so only
// magnitudes need block-local references (the paper's remark on log-decays and local
// renormalisation inside chunks, App. C.4).
//
// Pipeline (512 threads = 8 waves, two per SIMD; two barriers per step):
//   waves 0-3 (consumers) own 16 value columns each and hold their columns of the rotated
//     state in MFMA accumulators for the whole scan; they walk the four blocks of step s:
//       P = conj(K)G S,  O = conj(Q)G S,  Delta = N D_beta (conj(V) - P),  O += A Delta,
//       S <- |D| S + (K Q)^T Delta      (|D| the block's decay magnitude per channel);
//     after the middle barrier of step s each also forms block `wave` of step s + 1's
//     state-independent factors: the Gram matrices L and A on the matrix cores and the
//     inverse N = (I + D_beta L)^{-1} in fp32, beside its last block of step s;
//   waves 4-7 (producers) own one block of 16 tokens each.  Before the middle barrier they
//     form step s + 1's operands conj(Q)G, conj(K)G, k / P and K Q (bf16, to LDS) from
//     q, k requested a step earlier (a second register buffer) and request step s + 2's
//     q, k; after it they run step s + 2's prefix and suffix
//     decay products and phase sums (scans over a lane's four tokens and a wave's four
//     token segments; the phase offsets of earlier blocks through LDS) and request step
//     s + 3's alpha, theta.
//   Operands live in two LDS sets (steps s and s + 1).
//
// Complex products.  A complex 16 x 16 result block is held as two MFMA accumulator tiles,
// its real and its imaginary part (lane (c, g) holds row 4g + r, column c of each, r = 0..3).
// The left operand X is interleaved complex bf16 (lane word r = (Re, Im) of X[c][4g + r]);
// the right operand Y enters two MFMAs, one per output part:
//   real part:      B words (Re Y, -Im Y)        imaginary part:  B words (Im Y, Re Y)
// built in-lane (two converts from a split accumulator, or a sign flip and a half swap of
// an LDS word), so no lane exchange is needed anywhere in the state-dependent chain.  Four
// real multiply-adds per complex one (the real-coordinate view of Prop. 3.3), fp32
// accumulation.
//
// Global memory goes through buffer resources: every lane offset is fixed for the whole
// scan, the per-step part is folded into the resource base, and positions past the end of
// the sequence or past the last column read as zero (stores there are dropped), so the
// ragged tail needs no branches.
//
// LDS layouts.  A 64 x 64 complex bf16 array has rows padded from 256 to 272 bytes; a
// 16 x 16 complex bf16 block has 64-byte rows whose 16-byte chunks are XOR-swizzled by
// (row >> 2) & 3.  Either way one MFMA operand fragment (4 consecutive complex values of one
// row) is a single conflict-free 16-byte read.  conj(Q)G, conj(K)G and k_j / P_j are stored
// token-major (rows = tokens), K Q channel-major (rows = channels), each the layout its
// product reads as fragments.
#include <utility>

#include "sfda_device.h"
#include "sfda_launch.h"

namespace sfda {
namespace pipe {

constexpr int MP = 64;          // key channels per workgroup (m zero-padded)
constexpr int NTH = 512;
constexpr int CP = 64;          // tokens per pipeline step
constexpr int NB = CP / 16;     // 16-token blocks per step
constexpr int NB1 = 3;          // blocks the consumers walk before the step's middle barrier

typedef uint32_t u32;
typedef u32 u32x2 __attribute__((ext_vector_type(2)));
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

__device__ __forceinline__ bf16x8 as_bf(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }
typedef float f32x2 __attribute__((ext_vector_type(2)));
// two floats -> (lo, hi) bf16 pair, round to nearest even (one v_cvt_pk_bf16_f32)
__device__ __forceinline__ u32 pack_bf16(float lo, float hi) {
    const f32x2 v = {lo, hi};
    return __builtin_bit_cast(u32, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ float bf_lo(u32 w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(u32 w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(a), as_bf(b), c, 0, 0, 0);
}

// ------------------------------------------------------------------ complex MFMA operands

struct CAcc { f32x4 re, im; };     // split complex accumulator block
struct BPair { u32x4 re, im; };    // right operand for the real / imaginary output part

__device__ __forceinline__ void czero(CAcc& z) { z.re = zero4(); z.im = zero4(); }

// from interleaved complex bf16 words w[r] = (Re, Im) of Y[4g + r][c]
__device__ __forceinline__ BPair bwords(u32x4 w) {
    BPair b;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        b.re[r] = w[r] ^ 0x80000000u;
        b.im[r] = __builtin_amdgcn_alignbit(w[r], w[r], 16);
    }
    return b;
}

// from a split accumulator pair holding Y[4g + r][c]: (Re, -Im) and (Im, Re), each
// component rounded to bf16 once (the same bits as a sign flip and half swap of one pair)
__device__ __forceinline__ BPair bsplit(const CAcc& y) {
    BPair b;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        b.re[r] = pack_bf16(y.re[r], -y.im[r]);
        b.im[r] = pack_bf16(y.im[r], y.re[r]);
    }
    return b;
}

// z += X Y over one K-block of 16 complex indices
__device__ __forceinline__ void cmma(CAcc& z, u32x4 a, const BPair& b) {
    z.re = mfma(a, b.re, z.re);
    z.im = mfma(a, b.im, z.im);
}

// ------------------------------------------------------------------ buffer access

constexpr u32 OOB = 0x80000000u;     // lane offset that lies past every resource's range

// Every caller passes a wave-uniform size.  readfirstlane keeps it in a scalar register: a
// size the compiler had placed in a vector register (a max() does that) turns each load
// through the resource into a loop over the distinct descriptors of the wave.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, __builtin_amdgcn_readfirstlane(bytes),
                                             0x00020000);
}
__device__ __forceinline__ u32 ld16(rsrc_t r, u32 off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}
__device__ __forceinline__ u32 ld32(rsrc_t r, u32 off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ u32x2 ld64(rsrc_t r, u32 off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
}
__device__ __forceinline__ u32x4 ld128(rsrc_t r, u32 off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

template <typename TOUT> struct Out;
template <> struct Out<uint16_t> {      // complex bf16
    static constexpr int BYTES = 4;
    __device__ __forceinline__ static void store(rsrc_t r, u32 off, float re, float im) {
        __builtin_amdgcn_raw_buffer_store_b32(pack_bf16(re, im), r, off, 0, 0);
    }
};
template <> struct Out<float> {         // complex fp32
    static constexpr int BYTES = 8;
    __device__ __forceinline__ static void store(rsrc_t r, u32 off, float re, float im) {
        const u32x2 w = {__float_as_uint(re), __float_as_uint(im)};
        __builtin_amdgcn_raw_buffer_store_b64(w, r, off, 0, 0);
    }
};

// ------------------------------------------------------------------ lane exchange

// value of lane K of this lane's 16-lane row
template <int K>
__device__ __forceinline__ float row_lane(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x150 + K, 0xF, 0xF, false));
}
// quad permutation (DPP quad_perm selector P: lane i of a quad takes lane (P >> 2i) & 3).
// Call it where every lane of the wave is active (never as the unevaluated arm of a
// conditional expression): under a reduced exec mask a lane whose source lane is switched
// off reads the old register value instead of the source's data.
template <int P>
__device__ __forceinline__ float quad_lane(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), P, 0xF, 0xF, false));
}
// ------------------------------------------------------------------ LDS addressing (bytes)

// 64 x 64 complex bf16, row-major, rows padded to 272 bytes (68 words: consecutive rows start
// 4 banks apart, so 16 rows x one 16-byte chunk, or 16 consecutive words of 4 rows spaced
// 4 apart, touch distinct banks).  Offsets are linear in row and column, so every fragment
// address is one lane base plus an immediate.
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

// ------------------------------------------------------------------ 16 x 16 inverse

// N = (I - X)^{-1} for X strictly lower triangular (X = -(D_beta L) on a block), i.e.
// N = I + X N, by forward substitution over the pivots s = 0 .. 14.  Lane (i, cg) --
// i = lane % 16, cg = lane / 16 -- holds row i of X (zero on and above the diagonal, so
// rows i <= s take no update) and row i, columns cg, cg + 4, cg + 8, cg + 12 of N (slot k
// holds column 4k + cg); the pivot row N(s, .) is lane s of the lane's own 16-lane row (DPP
// row broadcast).  N is lower triangular, so the pivot row is zero past column s and slot
// k takes part only in the steps s >= 4k: 36 slot-steps instead of 60.
template <int S>
__device__ __forceinline__ void inv_step(float (&nr)[4], float (&ni)[4], const float2 (&xrow)[16])
{
    const float xr = xrow[S].x, xi = xrow[S].y;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (4 * k > S) continue;
        const float pr = row_lane<S>(nr[k]), pi = row_lane<S>(ni[k]);
        nr[k] = __builtin_fmaf(xr, pr, __builtin_fmaf(-xi, pi, nr[k]));
        ni[k] = __builtin_fmaf(xr, pi, __builtin_fmaf(xi, pr, ni[k]));
    }
}
template <int... S>
__device__ __forceinline__ void inv_steps(float (&nr)[4], float (&ni)[4], const float2 (&xrow)[16],
                                          std::integer_sequence<int, S...>)
{
    (inv_step<S>(nr, ni, xrow), ...);
}

// ------------------------------------------------------------------ shared memory

struct Smem {
    struct Set {
        u32x4 qb[CP * RP / 16];  // conj(q_t) e^{i phi_t} P_t         [token][channel]
        u32x4 kb[CP * RP / 16];  // conj(k_t) e^{i phi_t} P_t         [token][channel]
        u32x4 kr[MP * RP / 16];  // k_t e^{-i phi_t} Q_t              [channel][token]
        u32x4 nd[NB * 64];       // N_p = (I + D_beta L_p)^{-1}, one 16 x 16 block per block p
        u32x4 aq[NB * 64];       // A_p, lower triangle with the diagonal
        float dm[NB][MP];        // |D_p|: decay magnitude over block p, per channel
        int bad[NB];             // block p lies outside the decay range
    };
    Set set[2];
    u32x4 kd[CP * RP / 16];      // k_t e^{-i phi_t} / P_t (right operand of the blocks' Grams)
    float2 xs[NB][16][18];       // per producer wave: X of its block (fp32, padded)
    float tph[2][NB][MP];        // per block: theta / 2 pi summed over it, reduced to [0, 1)
    float2 rot[MP];              // e^{i phi} at the last token: the final state rotation
    float beta[3][CP];           // beta of step s at s % 3: written by the scans of step s
                                 // (two steps ahead), read by the factors and the steps
    u32 ostage[2][NB][256];      // o of consumer waves 0, 1 per block (complex bf16, token-major
                                 // 16 x 16), stored to global memory by waves 2, 3
};

struct Args {
    const uint16_t *q, *k, *v, *alpha, *theta, *beta;
    const float* S0;
    void* o;
    float* S_T;
    int T, m, n, n_slices, slice;
    // GATED: alpha = amin + aspan sigmoid(a), theta = tmax tanh(b), beta = sigmoid(c),
    // k = k~ / (||k~|| + eps) from the pre-activations passed in alpha, theta, beta, k
    float amin, aspan, tmax, eps;
};

// logistic function and tanh from the hardware exp2 and reciprocal (relative error a few
// ulp; saturate to 0 / 1 and -1 / 1 without NaN for large arguments)
__device__ __forceinline__ float sigmoid_f(float x) {
    return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}
__device__ __forceinline__ float tanh_f(float x) {
    return 1.f - 2.f * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(2.8853900817779268f * x));
}

template <typename TOUT, bool GATED>
__global__ __launch_bounds__(NTH, 1) void chunk_pipe_kernel(Args args)
{
    typedef Smem::Set Set;
    __shared__ Smem sm;

    const int T = args.T, m = args.m, n = args.n;
    long bh;
    int sl;
    head_slice(blockIdx.x, args.n_slices, gridDim.x / args.n_slices, bh, sl);
    const int n0 = sl * args.slice;
    const int scols = min(args.slice, n - n0);          // value columns of this slice
    const int nsteps = (T + CP - 1) / CP;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar)
    const int c = lane & 15;
    const int g = lane >> 4;
    const bool consumer = wave < 4;

    const long base_tm = bh * static_cast<long>(T) * m;
    const long base_tn = bh * static_cast<long>(T) * n;
    const long base_mn = bh * static_cast<long>(m) * n;
    const long base_t = bh * static_cast<long>(T);

    auto set_ptr = [&](int s) -> char* { return reinterpret_cast<char*>(&sm.set[s]); };
#ifdef SFDA_LDS_POISON
    // at the top of step st, by every wave: the operand set of step st + 1 (last read in step
    // st - 1), k / P and the inverse's scratch are rewritten before they are read
    auto poison_next = [&](int st) {
        lds_poison(&sm.set[(st + 1) & 1], sizeof(Set), tid, NTH);
        lds_poison(sm.kd, sizeof(sm.kd), tid, NTH);
        lds_poison(sm.xs, sizeof(sm.xs), tid, NTH);
        __syncthreads();
    };
#endif
    constexpr int OFF_QB = offsetof(Set, qb), OFF_KB = offsetof(Set, kb), OFF_KR = offsetof(Set, kr);
    constexpr int OFF_ND = offsetof(Set, nd), OFF_AQ = offsetof(Set, aq);

    if (consumer) {
        // ============================================================ consumer waves
        // wave w owns value columns n0 + 16 w .. n0 + 16 w + 15 of the slice
        const bool active = 16 * wave < scols;                   // wave-uniform
        const int jl = 16 * wave + c;
        const int jw = n0 + jl;
        const bool col_ok = jl < scols;
        u32 voff_v[4], voff_o[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const u32 e = static_cast<u32>((4 * g + r) * n + jw);
            voff_v[r] = col_ok ? e * 4u : OOB;
            voff_o[r] = col_ok ? e * static_cast<u32>(Out<TOUT>::BYTES) : OOB;
        }

        // v == NULL reads as zeros and o == NULL drops the stores: their ranges are empty
        // (an access outside a buffer range touches no memory)
        const int v_row_bytes = args.v ? n * 4 : 0;
        const int o_row_bytes = args.o ? n * Out<TOUT>::BYTES : 0;
        CAcc Sa[4];          // rotated state, rows kb*16 + 4g + r, column jw
        u32 vv[NB][4];       // v of the step in flight (complex bf16), prefetched
        // bf16 output: o of the step's blocks (complex bf16), stored together at the end of the
        // step.  A vector memory counter covers loads and stores in issue order, so a store
        // issued between a block's V prefetch and the next is waited for with that prefetch;
        // stored at the end of the step, every V prefetch of the step is older than them.
        constexpr bool OPACK = Out<TOUT>::BYTES == 4;
        u32 opk[NB][4];
        // A slice of exactly 32 columns leaves waves 2 and 3 without columns: then they do the
        // global memory traffic of waves 0 and 1 through an LDS slot per block, 16 bytes per
        // lane: load V into it before the block, store the o that waves 0 and 1 put into it
        // after (memory instructions cost the issuing wave; these two have time to spare).
        const bool staged = OPACK && scols == 32;                 // wave-uniform
        const bool helper = staged && wave >= 2;
        const int hw = wave - 2;                                 // the wave a helper stores for

        auto load_v = [&](int st, int p) {
            const int t0 = st * CP + p * 16;
            const rsrc_t rv = make_rsrc(args.v + 2 * (base_tn + static_cast<long>(t0) * n),
                                        max(T - t0, 0) * v_row_bytes);
#pragma unroll
            for (int r = 0; r < 4; ++r) vv[p][r] = ld32(rv, voff_v[r]);
        };

        TOUT* const go = static_cast<TOUT*>(args.o);
        auto consume = [&](int st, int p0, int p1) {
            const char* S = set_ptr(st & 1);
            const Set& ss = sm.set[st & 1];
            const int bad = __builtin_amdgcn_readfirstlane(ss.bad[0] | ss.bad[1] | ss.bad[2] | ss.bad[3]);
            if (p0 == 0 && bad) {
                const float nan = __builtin_nanf("");
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int r = 0; r < 4; ++r) { Sa[kb].re[r] = nan; Sa[kb].im[r] = nan; }
            }
#pragma unroll
            for (int p = 0; p < NB; ++p) {
                if (p < p0 || p >= p1) continue;
                const int t0 = st * CP + p * 16;
                // the state as right operands (channel blocks kb)
                BPair sb[4];
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) sb[kb] = bsplit(Sa[kb]);
                // P = conj(K)G S and O = conj(Q)G S over the block's 16 tokens
                CAcc R, O;
                czero(R);
                czero(O);
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const u32x4 ak = *reinterpret_cast<const u32x4*>(S + OFF_KB + rm_frag(p * 16 + c, kb * 4 + g));
                    const u32x4 aq = *reinterpret_cast<const u32x4*>(S + OFF_QB + rm_frag(p * 16 + c, kb * 4 + g));
                    cmma(R, ak, sb[kb]);
                    cmma(O, aq, sb[kb]);
                }
                // the state decays over the block: S <- |D_p| S (its operand form is taken)
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const float4 d4 = *reinterpret_cast<const float4*>(&ss.dm[p][kb * 16 + 4 * g]);
                    const float dr[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
                    for (int r = 0; r < 4; ++r) { Sa[kb].re[r] *= dr[r]; Sa[kb].im[r] *= dr[r]; }
                }
                // R = D_beta (conj(V) - P); staged: V of the block from the staging slot
                const float4 bt = *reinterpret_cast<const float4*>(&sm.beta[st % 3][p * 16 + 4 * g]);
                const float btr[4] = {bt.x, bt.y, bt.z, bt.w};
                if (staged) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) vv[p][r] = sm.ostage[wave][p][(4 * g + r) * 16 + c];
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const u32 w = vv[p][r];
                    R.re[r] = btr[r] * (bf_lo(w) - R.re[r]);
                    R.im[r] = -btr[r] * (bf_hi(w) + R.im[r]);
                }
                // this block's v is consumed: the next step's (past the last step an empty
                // range; issued every step so that every path through the loop has the same
                // loads in flight and the wait counts stay exact)
                if (!staged) load_v(st + 1, p);
                // Delta = N_p R
                const u32x4 fn = *reinterpret_cast<const u32x4*>(S + OFF_ND + p * 1024 + blk_frag(c, g));
                CAcc d;
                czero(d);
                cmma(d, fn, bsplit(R));
                const BPair db = bsplit(d);
                // O += A_p Delta; o = conj(O^*), rows past T and columns past the slice dropped
                const u32x4 fa = *reinterpret_cast<const u32x4*>(S + OFF_AQ + p * 1024 + blk_frag(c, g));
                cmma(O, fa, db);
                if constexpr (OPACK) {
                    if (staged) {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            sm.ostage[wave][p][(4 * g + r) * 16 + c] = pack_bf16(O.re[r], -O.im[r]);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r) opk[p][r] = pack_bf16(O.re[r], -O.im[r]);
                    }
                } else {
                    const rsrc_t ro = make_rsrc(go + 2 * (base_tn + static_cast<long>(t0) * n),
                                                max(T - t0, 0) * o_row_bytes);
#pragma unroll
                    for (int r = 0; r < 4; ++r) Out<TOUT>::store(ro, voff_o[r], O.re[r], -O.im[r]);
                }
                // S += (K Q)^T Delta: rows = channels kb*16 + c, K = the block's tokens
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const u32x4 f = *reinterpret_cast<const u32x4*>(S + OFF_KR + rm_frag(kb * 16 + c, p * 4 + g));
                    cmma(Sa[kb], f, db);
                }
            }
            if constexpr (OPACK) {
                if (p1 == NB && !staged) {
#pragma unroll
                    for (int p = 0; p < NB; ++p) {
                        const int t0 = st * CP + p * 16;
                        const rsrc_t ro = make_rsrc(go + 2 * (base_tn + static_cast<long>(t0) * n),
                                                    max(T - t0, 0) * o_row_bytes);
#pragma unroll
                        for (int r = 0; r < 4; ++r) __builtin_amdgcn_raw_buffer_store_b32(opk[p][r], ro, voff_o[r], 0, 0);
                    }
                }
            }
        };

        // a helper wave's store of block p of step s: lane L takes token L / 4, columns
        // 4 (L % 4) .. 4 (L % 4) + 3 of wave hw's 16 (rows past T are dropped by the range)
        auto hstore = [&](int s, int p) {
            const int t0 = s * CP + p * 16;
            const rsrc_t ro = make_rsrc(go + 2 * (base_tn + static_cast<long>(t0) * n),
                                        max(T - t0, 0) * o_row_bytes);
            const u32x4 w = *reinterpret_cast<const u32x4*>(&sm.ostage[hw][p][(lane >> 2) * 16 + 4 * (lane & 3)]);
            const u32 off = static_cast<u32>((lane >> 2) * n + n0 + 16 * hw + 4 * (lane & 3)) * 4u;
            __builtin_amdgcn_raw_buffer_store_b128(w, ro, off, 0, 0);
        };
        // ... and its load of wave hw's V for block p of step s (the same lane layout), put into
        // the block's slot once the slot's o has been stored: the slot then holds V until
        // wave hw reads it at the start of the block, and o after the block
        u32x4 hv[NB];
        auto hload = [&](int s, int p) {
            const int t0 = s * CP + p * 16;
            const rsrc_t rv = make_rsrc(args.v + 2 * (base_tn + static_cast<long>(t0) * n),
                                        max(T - t0, 0) * v_row_bytes);
            hv[p] = ld128(rv, static_cast<u32>((lane >> 2) * n + n0 + 16 * hw + 4 * (lane & 3)) * 4u);
        };
        auto hput = [&](int p) {
            *reinterpret_cast<u32x4*>(&sm.ostage[hw][p][(lane >> 2) * 16 + 4 * (lane & 3)]) = hv[p];
        };

        // block `wave` of step st: its Gram matrices L (strict lower) and A (with the diagonal)
        // and the inverse N = (I + D_beta L)^{-1}, from the operands the producers wrote before
        // the last barrier
        auto diag = [&](int st) {
            const int pw = wave;                 // this wave's block
            char* S = set_ptr(st & 1);
            const Set& ss = sm.set[st & 1];
            const char* KD = reinterpret_cast<const char*>(sm.kd);
            CAcc zl, za;
            czero(zl);
            czero(za);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                const u32x4 ak = *reinterpret_cast<const u32x4*>(S + OFF_KB + rm_frag(pw * 16 + c, kb * 4 + g));
                const u32x4 aq = *reinterpret_cast<const u32x4*>(S + OFF_QB + rm_frag(pw * 16 + c, kb * 4 + g));
                const u32x4 w = *reinterpret_cast<const u32x4*>(KD + rm_frag(pw * 16 + c, kb * 4 + g));
                const BPair bw = bwords(w);
                cmma(zl, ak, bw);
                cmma(za, aq, bw);
            }
            // A_p: lower triangle with the diagonal, zero above
            char* aqb = S + OFF_AQ + pw * 1024;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool keep = c <= 4 * g + r;
                *reinterpret_cast<u32*>(aqb + blk_off(4 * g + r, c)) = keep ? pack_bf16(za.re[r], za.im[r]) : 0u;
            }
            // X = -(D_beta L), zero on and above the diagonal, to the wave's scratch; each
            // lane then reads back one row
            const float4 bt = *reinterpret_cast<const float4*>(&sm.beta[st % 3][pw * 16 + 4 * g]);
            const float btr[4] = {bt.x, bt.y, bt.z, bt.w};
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool lo = c < 4 * g + r;
                sm.xs[pw][4 * g + r][c] = make_float2(lo ? -btr[r] * zl.re[r] : 0.f,
                                                      lo ? -btr[r] * zl.im[r] : 0.f);
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            const int i = c, cgi = g;
            float2 xrow[16];
#pragma unroll
            for (int s2 = 0; s2 < 16; s2 += 2) {
                const float4 x2 = *reinterpret_cast<const float4*>(&sm.xs[pw][i][s2]);
                xrow[s2] = make_float2(x2.x, x2.y);
                xrow[s2 + 1] = make_float2(x2.z, x2.w);
            }
            float nr[4], ni[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) { nr[k] = i == 4 * k + cgi ? 1.f : 0.f; ni[k] = 0.f; }
            inv_steps(nr, ni, xrow, std::make_integer_sequence<int, 15>{});
#pragma unroll
            for (int k = 0; k < 4; ++k)
                *reinterpret_cast<u32*>(S + OFF_ND + pw * 1024 + blk_off(i, 4 * k + cgi)) =
                    pack_bf16(nr[k], ni[k]);
        };

        // The role test is wave-uniform and encloses each role's whole life (prologue, step
        // loop, epilogue), so each role keeps only its own registers live.  Both loops pass
        // the same sequence of workgroup barriers: two per step plus the lead-in.
        if (active) {
            const rsrc_t rs = make_rsrc(args.S0 ? args.S0 + 2 * base_mn : args.S0,
                                        args.S0 ? m * n * 8 : 0);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = kb * 16 + 4 * g + r;
                    const u32 off = (col_ok && i < m) ? static_cast<u32>(i * n + jw) * 8u : OOB;
                    const u32x2 x = ld64(rs, off);
                    Sa[kb].re[r] = __uint_as_float(x.x);
                    Sa[kb].im[r] = __uint_as_float(x.y);
                }
            if (nsteps > 0 && !staged) {
#pragma unroll
                for (int p = 0; p < NB; ++p) load_v(0, p);
            }
        }
        __syncthreads();          // matches the producers' lead-in barrier
        for (int st = -1; st < nsteps; ++st) {
#ifdef SFDA_LDS_POISON
            poison_next(st);
#endif
            // phase 1: the first NB1 blocks of step st (the producers form step st + 1's operands)
            if (helper) {                            // V of the next step's first blocks
#pragma unroll
                for (int p = 0; p < NB1; ++p) hload(st + 1, p);
            }
            if (active && st >= 0) consume(st, 0, NB1);
            if (helper) {                            // the previous step's last blocks: o out, V in
#pragma unroll
                for (int p = NB1; p < NB; ++p) {
                    if (st >= 1) hstore(st - 1, p);
                    if (st >= 0) hput(p);
                }
            }
            __syncthreads();
            // phase 2: this wave's block of step st + 1 (Grams, inverse), the rest of step st
            if (helper) {                            // V of the next step's last blocks
#pragma unroll
                for (int p = NB1; p < NB; ++p) hload(st + 1, p);
            }
            if (st + 1 < nsteps) diag(st + 1);
            if (active && st >= 0) consume(st, NB1, NB);
            if (helper) {                            // this step's first blocks: o out, V in
#pragma unroll
                for (int p = 0; p < NB1; ++p) {
                    if (st >= 0) hstore(st, p);
                    hput(p);
                }
            }
            __syncthreads();
        }
        if (helper && nsteps > 0) {
#pragma unroll
            for (int p = NB1; p < NB; ++p) hstore(nsteps - 1, p);
        }
        if (active && args.S_T != nullptr) {
            // back from the rotated frame: S_T = diag(e^{i phi_T}) S
            const rsrc_t rs = make_rsrc(args.S_T + 2 * base_mn, m * n * 8);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = kb * 16 + 4 * g + r;
                    const u32 off = (col_ok && i < m) ? static_cast<u32>(i * n + jw) * 8u : OOB;
                    float sr = Sa[kb].re[r], si = Sa[kb].im[r];
                    if (nsteps > 0) {
                        const float2 z = sm.rot[i];
                        const float tr = __builtin_fmaf(z.x, sr, -z.y * si);
                        si = __builtin_fmaf(z.x, si, z.y * sr);
                        sr = tr;
                    }
                    const u32x2 w = {__float_as_uint(sr), __float_as_uint(si)};
                    __builtin_amdgcn_raw_buffer_store_b64(w, rs, off, 0, 0);
                }
        }
    } else {
        // ============================================================ producer waves
        // Wave pw owns block pw (tokens 16 pw .. 16 pw + 15) of every step for all channels, so
        // one load instruction covers whole rows of q, k, alpha, theta (whole cache lines).
        // Lane = (channel group cg: channels 4cg .. 4cg+3; token segment tsg: 4 tokens).
        const int pw = wave - 4;
        const int tsg = lane & 3;
        const int cg = lane >> 2;
        const int pc0 = cg * 4;                        // first of this lane's 4 channels
        const int tl0 = pw * 16 + tsg * 4;             // first token (in the step) of the lane
        const bool wide = (m & 3) == 0;               // 4-channel vector loads
        u32 poff2[4], poff4[4];                       // byte offsets (bf16 / complex bf16)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const u32 e = static_cast<u32>((tl0 + u) * m + pc0);
            poff2[u] = pc0 < m ? e * 2u : OOB;
            poff4[u] = pc0 < m ? e * 4u : OOB;
        }
        uint2 pa[4], pt[4];               // alpha, theta of the 4 channels (bf16 pairs)
        u32 pb;                           // beta of the block's tokens (lanes 0..15)
        // q, k of the 4 channels (complex bf16) of one step; two of them, so that a step's q
        // and k are requested a whole step before their operands are formed (global loads take
        // several thousand cycles under this load); the copy waits for loads issued a step
        // earlier
        struct QK { u32x4 q[4], k[4]; };
        QK cur, nxt;

        // alpha, theta, beta of step st (consumed by the scan, a step before the rest)
        auto load_at = [&](int st, auto wide_c) __attribute__((always_inline)) {
            const int t0 = st * CP;
            const long e0 = base_tm + static_cast<long>(t0) * m;
            const int rows = max(T - t0, 0);      // past the last step: an empty range
            const rsrc_t ra = make_rsrc(args.alpha + e0, rows * m * 2);
            const rsrc_t rt = make_rsrc(args.theta + e0, rows * m * 2);
            if constexpr (decltype(wide_c)::value) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const u32x2 a = ld64(ra, poff2[u]), t = ld64(rt, poff2[u]);
                    pa[u] = make_uint2(a.x, a.y);
                    pt[u] = make_uint2(t.x, t.y);
                }
            } else {                    // any m: one channel per load
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    u32 a4[4], t4[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const u32 e = static_cast<u32>((tl0 + u) * m + pc0 + k);
                        const bool ok = pc0 + k < m;
                        a4[k] = ld16(ra, ok ? e * 2u : OOB);
                        t4[k] = ld16(rt, ok ? e * 2u : OOB);
                    }
                    pa[u] = make_uint2(a4[0] | (a4[1] << 16), a4[2] | (a4[3] << 16));
                    pt[u] = make_uint2(t4[0] | (t4[1] << 16), t4[2] | (t4[3] << 16));
                }
            }
            const rsrc_t rb = make_rsrc(args.beta + base_t + t0, rows * 2);
            pb = ld16(rb, lane < 16 ? static_cast<u32>(pw * 16 + lane) * 2u : OOB);
        };
        // q, k of step st
        auto load_qk = [&](int st, QK& b, auto wide_c) __attribute__((always_inline)) {
            const int t0 = st * CP;
            const long e0 = base_tm + static_cast<long>(t0) * m;
            const int rows = max(T - t0, 0);      // past the last step: an empty range
            const rsrc_t rq = make_rsrc(args.q + 2 * e0, rows * m * 4);
            const rsrc_t rk = make_rsrc(args.k + 2 * e0, rows * m * 4);
            if constexpr (decltype(wide_c)::value) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    b.q[u] = ld128(rq, poff4[u]);
                    b.k[u] = ld128(rk, poff4[u]);
                }
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u)
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const u32 e = static_cast<u32>((tl0 + u) * m + pc0 + k);
                        const bool ok = pc0 + k < m;
                        b.q[u][k] = ld32(rq, ok ? e * 4u : OOB);
                        b.k[u][k] = ld32(rk, ok ? e * 4u : OOB);
                    }
            }
        };

        // Scans of one block per channel (three levels: the lane's 4 tokens, the wave's four
        // segments by quad DPP, and for the phase the earlier blocks through LDS):
        //   P_t = prod of alpha from the block's first token to t    (forwards, <= 1)
        //   Q_t = prod of alpha from t + 1 to the block's last token (backwards, <= 1)
        //   phi_t = sum of theta / 2 pi up to t, reduced to [0, 1) revolutions
        // Positions past T or past m are identity tokens (alpha = 1, theta = 0).
        constexpr float INV_2PI = 0.15915494309189535f;
        float Pf[4][4], Qb[4][4], ph[4][4];   // [token u][channel k] of the lane
        float dtot[4], invd[4];               // block decay magnitude D and 1 / D per channel
        int oor = 0;                          // a channel of the block decays below 2^-126
        auto pretot_body = [&](int st, auto padded) __attribute__((always_inline)) {
            const bool s0 = tsg == 0, s01 = tsg < 2, s3 = tsg == 3, s23 = tsg >= 2;
            float tpk[4];
            bool low = false;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                float a[4], lp[4];
                float rp = 0.f;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const u32 wa = k < 2 ? pa[u].x : pa[u].y;
                    const u32 wt = k < 2 ? pt[u].x : pt[u].y;
                    float av = (k & 1) ? bf_hi(wa) : bf_lo(wa);
                    float th = (k & 1) ? bf_hi(wt) : bf_lo(wt);
                    if constexpr (GATED) {
                        av = args.amin + args.aspan * sigmoid_f(av);
                        th = args.tmax * tanh_f(th);
                    }
                    if constexpr (decltype(padded)::value) {
                        const bool ok = st * CP + tl0 + u < T && pc0 + k < m;
                        av = ok ? av : 1.f;
                        th = ok ? th : 0.f;
                    }
                    a[u] = av;
                    rp = __builtin_amdgcn_fractf(__builtin_fmaf(th, INV_2PI, rp));
                    lp[u] = rp;
                }
                // lane level: inclusive prefix and exclusive suffix of alpha
                const float m0 = a[0], m1 = m0 * a[1], m2 = m1 * a[2], m3 = m2 * a[3];
                const float x2 = a[3], x1 = a[2] * a[3], x0 = a[1] * x1;
                // quad level over the segments: exclusive prefix (earlier segments) and
                // exclusive suffix (later segments) of the segment products, phase prefix
                float im = m3, ip = rp, is = m3;
                float y = quad_lane<0x90>(im), yp = quad_lane<0x90>(ip);       // [0, 0, 1, 2]
                im *= s0 ? 1.f : y;
                ip += s0 ? 0.f : yp;
                y = quad_lane<0x40>(im); yp = quad_lane<0x40>(ip);             // [0, 0, 0, 1]
                im *= s01 ? 1.f : y;
                ip += s01 ? 0.f : yp;
                float ys = quad_lane<0xF9>(is);                                // [1, 2, 3, 3]
                is *= s3 ? 1.f : ys;
                ys = quad_lane<0xFE>(is);                                      // [2, 3, 3, 3]
                is *= s23 ? 1.f : ys;
                // every lane takes part in each move; the selects come after
                const float pm = quad_lane<0x90>(im), pp = quad_lane<0x90>(ip);
                const float ps = quad_lane<0xF9>(is);
                const float D = quad_lane<0xFF>(im), pt3 = quad_lane<0xFF>(ip);   // [3, 3, 3, 3]
                const float em = s0 ? 1.f : pm;                                // exclusive prefix
                const float ep = s0 ? 0.f : pp;
                const float es = s3 ? 1.f : ps;                                // exclusive suffix
                tpk[k] = __builtin_amdgcn_fractf(pt3);
                Pf[0][k] = em * m0; Pf[1][k] = em * m1; Pf[2][k] = em * m2; Pf[3][k] = em * m3;
                if constexpr (!GATED) { Qb[0][k] = es * x0; Qb[1][k] = es * x1; Qb[2][k] = es * x2; Qb[3][k] = es; }
#pragma unroll
                for (int u = 0; u < 4; ++u) ph[u][k] = ep + lp[u];
                dtot[k] = D;
                invd[k] = __builtin_amdgcn_rcpf(D);
                low = low || !(D >= 1.17549435e-38f);          // below the normal range (or NaN)
            }
            oor = __builtin_amdgcn_readfirstlane(static_cast<int>(__builtin_amdgcn_ballot_w64(low) != 0));
            if (s0) {
                float4* tw = reinterpret_cast<float4*>(&sm.tph[st & 1][pw][pc0]);
                tw[0] = make_float4(tpk[0], tpk[1], tpk[2], tpk[3]);
            }
        };

        // scans of step st (inputs in pa, pt), the block's phase total to LDS.  Only a step
        // with padding (ragged tail, m < 64) needs the identity-token substitution.
        auto pretot = [&](int st) __attribute__((always_inline)) {
            if ((st + 1) * CP <= T && m == MP) pretot_body(st, std::false_type{});
            else pretot_body(st, std::true_type{});
            if (lane < 16) {
                float bt = bf16_bits_to_f32(static_cast<uint16_t>(pb));
                if constexpr (GATED) bt = st * CP + pw * 16 + lane < T ? sigmoid_f(bt) : 0.f;
                sm.beta[st % 3][pw * 16 + lane] = bt;
            }
        };

        float base[4] = {0.f, 0.f, 0.f, 0.f};   // phase (revolutions) before the step, per channel

        // operands of step st into set st & 1: conj(Q)G, conj(K)G, K Q and the Gram operand
        auto produce = [&](int st, const QK& b) __attribute__((always_inline)) {
            char* S = set_ptr(st & 1);
            Set& ss = sm.set[st & 1];
            float off[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) off[k] = base[k];
            for (int w2 = 0; w2 < pw; ++w2) {          // phases of the earlier blocks
                const float4 t4 = *reinterpret_cast<const float4*>(&sm.tph[st & 1][w2][pc0]);
                off[0] += t4.x; off[1] += t4.y; off[2] += t4.z; off[3] += t4.w;
            }
            // GATED: 1 / (||k~_t|| + eps) of the lane's tokens; a token row lives on the 16
            // lanes tsg + 4 cg (four per 16-lane row): rotate by 4 and 8 inside the row, then
            // exchange across rows
            float kinv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                kinv[u] = 1.f;
                if constexpr (GATED) {
                    float s2 = 0.f;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const float kr = bf_lo(b.k[u][k]), ki = bf_hi(b.k[u][k]);
                        s2 = __builtin_fmaf(kr, kr, __builtin_fmaf(ki, ki, s2));
                    }
                    s2 += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s2), 0x124, 0xF, 0xF, false));
                    s2 += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s2), 0x128, 0xF, 0xF, false));
                    s2 += __shfl_xor(s2, 16);
                    s2 += __shfl_xor(s2, 32);
                    const float den = __builtin_sqrtf(s2) + args.eps;
                    kinv[u] = den > 0.f ? __builtin_amdgcn_rcpf(den) : 0.f;
                }
            }
            const bool last = st == nsteps - 1 && pw == NB - 1 && tsg == 3;
            u32 krw[4][4];                       // [channel k][token u]
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int tl = tl0 + u;
                u32x4 wq, wk, wd;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const float Ph = off[k] + ph[u][k];
                    const float sn = __builtin_amdgcn_sinf(Ph), cs = __builtin_amdgcn_cosf(Ph);
                    const u32 qw = b.q[u][k], kw = b.k[u][k];
                    const float qr = bf_lo(qw), qi = bf_hi(qw), kr = bf_lo(kw), ki = bf_hi(kw);
                    // conj(q) e^{i phi}, conj(k) e^{i phi}; k e^{-i phi} is the latter's conjugate
                    const float qur = __builtin_fmaf(qr, cs, qi * sn), qui = __builtin_fmaf(qr, sn, -qi * cs);
                    const float kur = __builtin_fmaf(kr, cs, ki * sn), kui = __builtin_fmaf(kr, sn, -ki * cs);
                    const float P = Pf[u][k];
                    // gated: Q_t = D / P_t (alpha >= alpha_min keeps P_t a normal float), which
                    // frees the suffix products' registers
                    const float Qt = GATED ? dtot[k] * __builtin_amdgcn_rcpf(P) : Qb[u][k];
                    const float Pk = P * kinv[u], Qk = Qt * kinv[u];
                    const float Dk = Qk * invd[k];             // 1 / P_t (= Q_t / D), times kinv
                    wq[k] = pack_bf16(qur * P, qui * P);
                    wk[k] = pack_bf16(kur * Pk, kui * Pk);
                    wd[k] = pack_bf16(kur * Dk, -kui * Dk);
                    krw[k][u] = pack_bf16(kur * Qk, -kui * Qk);
                    if (last && u == 3) sm.rot[pc0 + k] = make_float2(cs, sn);
                }
                *reinterpret_cast<u32x4*>(S + OFF_QB + rm_off(tl, pc0)) = wq;
                *reinterpret_cast<u32x4*>(S + OFF_KB + rm_off(tl, pc0)) = wk;
                *reinterpret_cast<u32x4*>(reinterpret_cast<char*>(sm.kd) + rm_off(tl, pc0)) = wd;
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const u32x4 w = {krw[k][0], krw[k][1], krw[k][2], krw[k][3]};
                *reinterpret_cast<u32x4*>(S + OFF_KR + rm_off(pc0 + k, tl0)) = w;
            }
            // the phase reached after the step, for the next one
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                float tot = base[k];
#pragma unroll
                for (int w2 = 0; w2 < NB; ++w2) tot += sm.tph[st & 1][w2][pc0 + k];
                base[k] = __builtin_amdgcn_fractf(tot);
            }
            if (tsg == 0) *reinterpret_cast<float4*>(&ss.dm[pw][pc0]) = make_float4(dtot[0], dtot[1], dtot[2], dtot[3]);
            if (lane == 0) ss.bad[pw] = oor;
        };

        // The step loop is instantiated once per load shape (4-channel vector loads, or one
        // channel per load for m not a multiple of 4), so that every path through one
        // instance issues the same loads and the compiler's wait counts stay exact.
        auto run = [&](auto wide_c) __attribute__((always_inline)) {
            if (nsteps > 0) {
                load_at(0, wide_c);
                load_qk(0, nxt, wide_c);
                pretot(0);
                if (nsteps > 1) load_at(1, wide_c);
            }
            __syncthreads();          // block phase totals of step 0
            for (int st = -1; st < nsteps; ++st) {
#ifdef SFDA_LDS_POISON
                poison_next(st);
#endif
                // phase 1: the operands of step st + 1 (q, k requested a step ago), the next
                // q, k.  The loads are issued on every step (past the last step their ranges
                // are empty): a path without them would make the wait counts at the loop head
                // cover the younger alpha, theta and beta loads too.  (The gated variant's
                // scans hold more registers; with the second buffer a few are spilled, which
                // costs less than requesting q, k only once the operands are formed.)
                if (st + 1 < nsteps) cur = nxt;
                load_qk(st + 2, nxt, wide_c);
                if (st + 1 < nsteps) produce(st + 1, cur);
                __syncthreads();
                // phase 2: the scans of step st + 2, alpha, theta and beta of the step after
                if (st + 2 < nsteps) pretot(st + 2);
                load_at(st + 3, wide_c);
                __syncthreads();
            }
        };
        if (wide) run(std::true_type{});
        else run(std::false_type{});
        // The compiler joins the two roles' control flow after the producer's exit, and the
        // wait-count analysis then treats the producer's last loads as in flight inside the
        // consumer loop; clearing them here keeps that loop from waiting on its own V loads.
        __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
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
    a.amin = L.alpha_min; a.aspan = L.alpha_max - L.alpha_min; a.tmax = L.theta_max; a.eps = L.eps;
    const dim3 grid(static_cast<unsigned>(static_cast<long>(L.B) * L.H * a.n_slices));
    if (L.gated) hipLaunchKernelGGL((chunk_pipe_kernel<TOUT, true>), grid, dim3(NTH), 0, st, a);
    else hipLaunchKernelGGL((chunk_pipe_kernel<TOUT, false>), grid, dim3(NTH), 0, st, a);
    return hipGetLastError();
}

}  // namespace pipe

hipError_t launch_chunk_bf16(const ChunkLaunch& L, hipStream_t st)
{
    return L.out_bf16 ? pipe::launch_t<uint16_t>(L, st) : pipe::launch_t<float>(L, st);
}

}  // namespace sfda
