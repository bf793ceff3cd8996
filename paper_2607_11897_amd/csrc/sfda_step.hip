// Recurrent decode step of SFDA (Sec. 3, Eq. (sfda) and the readout o = S^* q), one token
// per (batch, head), state updated in place.
//
// Per head, with S' = Lambda S (row i scaled by lambda_i = alpha_i e^{i theta_i}):
//   a = k^* S'            (1 x n)      b = q^* S'            (1 x n)
//   delta = beta (conj(v) - a)          so S = S' + k delta  (= (I - beta k k^*) S' + beta k v^*)
//   o = S^* q = conj(b + (q^* k) delta)
// which reads S once and writes it once -- the step is bound by HBM bandwidth.
//
// Launch: one 256-thread workgroup per (head, slice of NP value columns); NP is a power of
// two <= 64.  Thread (rg, j) owns column j (for even n: the column pair 2j, 2j + 1, so every
// state access is 16 bytes) and rows rg, rg + G, rg + 2G, ... (G = 256 / threads per row),
// so each wave reads and writes whole contiguous row segments.  The state is read and
// written with non-temporal accesses (it is streamed once per step), and the pair kernel is
// held to 64 VGPRs so that 8 waves share each SIMD: together these took the step from
// 5.3 to 5.9 TB/s of state traffic (with cached stores it stays near 5.3 at any occupancy).
// Column sums over rows are reduced in a fixed order through LDS (deterministic; no atomics).
#include "sfda_device.h"
#include "sfda_launch.h"

namespace sfda {

template <typename TIN, typename TOUT, int NP>
__global__ __launch_bounds__(256) void step_kernel(
    const TIN* __restrict__ q, const TIN* __restrict__ k, const TIN* __restrict__ v,
    const TIN* __restrict__ alpha, const TIN* __restrict__ theta, const TIN* __restrict__ beta,
    float* __restrict__ S, TOUT* __restrict__ o, int m, int n, int n_slices)
{
    constexpr int G = 256 / NP;                 // row groups
    constexpr int RPT = (64 + G - 1) / G;       // rows per thread (m <= 64)
    const long bh = blockIdx.x / n_slices;
    const int sl = blockIdx.x - static_cast<int>(bh) * n_slices;
    const int tid = threadIdx.x;
    const int jl = tid % NP;
    const int rg = tid / NP;
    const int j = sl * NP + jl;
    const bool colok = j < n;

    __shared__ float2 lam_s[64], k_s[64], q_s[64];
    __shared__ float2 red_a[G][NP], red_b[G][NP];
    __shared__ float2 delta_s[NP];
    __shared__ float2 qk_s;

    // state loads first, so their latency overlaps the small per-head set-up below
    float* Sh = S + bh * m * n * 2;
    float2 s[RPT];
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const int i = rg + G * r;
        s[r] = (i < m && colok) ? *reinterpret_cast<const float2*>(Sh + 2 * (static_cast<long>(i) * n + j))
                                : make_float2(0.f, 0.f);
    }

    if (tid < 64) {
        float2 qk = make_float2(0.f, 0.f);
        if (tid < m) {
            const long e = bh * m + tid;
            const float a = Elem<TIN>::load(alpha, e);
            float sn, cs;
            sincosf(Elem<TIN>::load(theta, e), &sn, &cs);
            lam_s[tid] = make_float2(a * cs, a * sn);
            const float2 kk = Elem<TIN>::load2(k, e);
            const float2 qq = Elem<TIN>::load2(q, e);
            k_s[tid] = kk;
            q_s[tid] = qq;
            qk = make_float2(qq.x * kk.x + qq.y * kk.y, qq.x * kk.y - qq.y * kk.x);  // conj(q) k
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            qk.x += __shfl_xor(qk.x, off);
            qk.y += __shfl_xor(qk.y, off);
        }
        if (tid == 0) qk_s = qk;
    }
    __syncthreads();

    // S' = Lambda S and the column partial sums a = k^* S', b = q^* S'
    float2 pa = make_float2(0.f, 0.f), pb = make_float2(0.f, 0.f);
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const int i = rg + G * r;
        if (i < m) {
            const float2 l = lam_s[i];
            const float2 x = s[r];
            const float2 y = make_float2(l.x * x.x - l.y * x.y, l.x * x.y + l.y * x.x);
            s[r] = y;
            const float2 kk = k_s[i];
            const float2 qq = q_s[i];
            pa.x += kk.x * y.x + kk.y * y.y;
            pa.y += kk.x * y.y - kk.y * y.x;
            pb.x += qq.x * y.x + qq.y * y.y;
            pb.y += qq.x * y.y - qq.y * y.x;
        }
    }
    red_a[rg][jl] = pa;
    red_b[rg][jl] = pb;
    __syncthreads();

    if (rg == 0) {
        float2 a = make_float2(0.f, 0.f), b = make_float2(0.f, 0.f);
#pragma unroll
        for (int gi = 0; gi < G; ++gi) {
            a.x += red_a[gi][jl].x; a.y += red_a[gi][jl].y;
            b.x += red_b[gi][jl].x; b.y += red_b[gi][jl].y;
        }
        float2 d = make_float2(0.f, 0.f);
        if (colok) {
            const float bt = Elem<TIN>::load(beta, bh);
            const float2 vv = Elem<TIN>::load2(v, bh * n + j);
            d = make_float2(bt * (vv.x - a.x), bt * (-vv.y - a.y));
            const float2 qk = qk_s;
            const float2 ob = make_float2(b.x + qk.x * d.x - qk.y * d.y, b.y + qk.x * d.y + qk.y * d.x);
            Elem<TOUT>::store2(o, bh * n + j, ob.x, -ob.y);
        }
        delta_s[jl] = d;
    }
    __syncthreads();

    const float2 d = delta_s[jl];
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const int i = rg + G * r;
        if (i < m && colok) {
            const float2 kk = k_s[i];
            const float2 x = s[r];
            *reinterpret_cast<float2*>(Sh + 2 * (static_cast<long>(i) * n + j)) =
                make_float2(x.x + kk.x * d.x - kk.y * d.y, x.y + kk.x * d.y + kk.y * d.x);
        }
    }
}

// Column-pair variant for even n: thread (rg, jp) owns columns 2 jp, 2 jp + 1 of the slice.
// Row block r (rows r G .. r G + G - 1) is addressed through a buffer resource of its own
// that starts at row r G and ends at row m, so one 32-bit lane offset (row rg, column j)
// serves every block and the per-row addresses live in scalar registers (the caller keeps
// n below 2^22, so the offsets stay under 2^31).  Rows past m lie past their resource's
// range: their loads return zero and their stores are dropped, and zero gates, keys and
// queries for those rows make them contribute nothing.  Columns past n (a ragged last
// slice) get a lane offset past every range.
typedef float f32v4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32v4 __attribute__((ext_vector_type(4)));
constexpr uint32_t STEP_OOB = 0x80000000u;
constexpr int STEP_NT = 2;          // buffer cache policy: non-temporal

template <typename TIN, typename TOUT, int NP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(8, 8))) void step_pair_kernel(
    const TIN* __restrict__ q, const TIN* __restrict__ k, const TIN* __restrict__ v,
    const TIN* __restrict__ alpha, const TIN* __restrict__ theta, const TIN* __restrict__ beta,
    float* __restrict__ S, TOUT* __restrict__ o, int m, int n, int n_slices)
{
    constexpr int NPR = NP / 2;                  // column pairs per workgroup
    constexpr int G = 256 / NPR;                 // row groups
    constexpr int RPT = (64 + G - 1) / G;        // rows per thread (m <= 64)
    constexpr int MR = G * RPT;                  // rows covered, m <= MR <= 256
    const long bh = blockIdx.x / n_slices;
    const int sl = blockIdx.x - static_cast<int>(bh) * n_slices;
    const int tid = threadIdx.x;
    const int jp = tid % NPR;
    const int rg = tid / NPR;
    const int j = sl * NP + 2 * jp;              // first column of the pair
    const bool colok = j < n;                    // n even: j + 1 < n as well

    __shared__ float2 lam_s[MR], k_s[MR], q_s[MR];
    __shared__ float4 red_a[G][NPR], red_b[G][NPR];
    __shared__ float4 delta_s[NPR];
    __shared__ float2 qk_s;

    float* Sh = S + bh * m * n * 2;
    auto block_rsrc = [&](int r) {
        const int rows = m - G * r;
        return __builtin_amdgcn_make_buffer_rsrc(Sh + static_cast<long>(G * r) * n * 2, 0,
                                                 rows > 0 ? rows * n * 8 : 0, 0x00020000);
    };
    const uint32_t off0 = colok ? static_cast<uint32_t>(rg * n + j) * 8u : STEP_OOB;
    f32v4 s[RPT];
#pragma unroll
    for (int r = 0; r < RPT; ++r)
        s[r] = __builtin_bit_cast(f32v4, __builtin_amdgcn_raw_buffer_load_b128(block_rsrc(r), off0, 0, STEP_NT));

    if (tid < MR) {
        float2 lam = make_float2(0.f, 0.f), kk = lam, qq = lam;
        if (tid < m) {
            const long e = bh * m + tid;
            const float a = Elem<TIN>::load(alpha, e);
            float sn, cs;
            sincosf(Elem<TIN>::load(theta, e), &sn, &cs);
            lam = make_float2(a * cs, a * sn);
            kk = Elem<TIN>::load2(k, e);
            qq = Elem<TIN>::load2(q, e);
        }
        lam_s[tid] = lam;
        k_s[tid] = kk;
        q_s[tid] = qq;
        if (tid < 64) {
            float2 qk = make_float2(qq.x * kk.x + qq.y * kk.y, qq.x * kk.y - qq.y * kk.x);  // conj(q) k
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                qk.x += __shfl_xor(qk.x, off);
                qk.y += __shfl_xor(qk.y, off);
            }
            if (tid == 0) qk_s = qk;
        }
    }
    __syncthreads();

    // S' = Lambda S and the column partial sums a = k^* S', b = q^* S' (both columns)
    float4 pa = make_float4(0.f, 0.f, 0.f, 0.f), pb = pa;
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const int i = rg + G * r;
        const float2 l = lam_s[i], kk = k_s[i], qq = q_s[i];
        const f32v4 x = s[r];
        const f32v4 y = {l.x * x.x - l.y * x.y, l.x * x.y + l.y * x.x,
                         l.x * x.z - l.y * x.w, l.x * x.w + l.y * x.z};
        s[r] = y;
        pa.x += kk.x * y.x + kk.y * y.y; pa.y += kk.x * y.y - kk.y * y.x;
        pa.z += kk.x * y.z + kk.y * y.w; pa.w += kk.x * y.w - kk.y * y.z;
        pb.x += qq.x * y.x + qq.y * y.y; pb.y += qq.x * y.y - qq.y * y.x;
        pb.z += qq.x * y.z + qq.y * y.w; pb.w += qq.x * y.w - qq.y * y.z;
    }
    red_a[rg][jp] = pa;
    red_b[rg][jp] = pb;
    __syncthreads();

    if (rg == 0) {
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
#pragma unroll 2
        for (int gi = 0; gi < G; ++gi) {
            const float4 x = red_a[gi][jp], y = red_b[gi][jp];
            a.x += x.x; a.y += x.y; a.z += x.z; a.w += x.w;
            b.x += y.x; b.y += y.y; b.z += y.z; b.w += y.w;
        }
        float4 d = make_float4(0.f, 0.f, 0.f, 0.f);
        if (colok) {
            const float bt = Elem<TIN>::load(beta, bh);
            const float2 v0 = Elem<TIN>::load2(v, bh * n + j), v1 = Elem<TIN>::load2(v, bh * n + j + 1);
            d = make_float4(bt * (v0.x - a.x), bt * (-v0.y - a.y), bt * (v1.x - a.z), bt * (-v1.y - a.w));
            const float2 qk = qk_s;
            const float4 ob = make_float4(b.x + qk.x * d.x - qk.y * d.y, b.y + qk.x * d.y + qk.y * d.x,
                                          b.z + qk.x * d.z - qk.y * d.w, b.w + qk.x * d.w + qk.y * d.z);
            Elem<TOUT>::store2(o, bh * n + j, ob.x, -ob.y);
            Elem<TOUT>::store2(o, bh * n + j + 1, ob.z, -ob.w);
        }
        delta_s[jp] = d;
    }
    __syncthreads();

    const float4 d = delta_s[jp];
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const float2 kk = k_s[rg + G * r];
        const f32v4 x = s[r];
        const f32v4 y = {x.x + kk.x * d.x - kk.y * d.y, x.y + kk.x * d.y + kk.y * d.x,
                         x.z + kk.x * d.z - kk.y * d.w, x.w + kk.x * d.w + kk.y * d.z};
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32v4, y), block_rsrc(r), off0, 0, STEP_NT);
    }
}

template <typename TIN, typename TOUT>
static hipError_t launch_step_t(const StepLaunch& L, hipStream_t st)
{
    int np = 1;
    while (np < L.n && np < 64) np <<= 1;
    const int n_slices = (L.n + np - 1) / np;
    const dim3 grid(static_cast<unsigned>(static_cast<long>(L.B) * L.H * n_slices));
    const TIN* q = static_cast<const TIN*>(L.q);
    const TIN* k = static_cast<const TIN*>(L.k);
    const TIN* v = static_cast<const TIN*>(L.v);
    const TIN* a = static_cast<const TIN*>(L.alpha);
    const TIN* th = static_cast<const TIN*>(L.theta);
    const TIN* b = static_cast<const TIN*>(L.beta);
    TOUT* o = static_cast<TOUT*>(L.o);
#define SFDA_STEP_CASE(NP_)                                                              \
    case NP_:                                                                            \
        hipLaunchKernelGGL((step_kernel<TIN, TOUT, NP_>), grid, dim3(256), 0, st, q, k, v, a, \
                           th, b, L.S, o, L.m, L.n, n_slices);                           \
        break;
#define SFDA_STEP_PAIR_CASE(NP_)                                                         \
    case NP_:                                                                            \
        hipLaunchKernelGGL((step_pair_kernel<TIN, TOUT, NP_>), grid, dim3(256), 0, st, q, k, v, \
                           a, th, b, L.S, o, L.m, L.n, n_slices);                        \
        break;
    if ((L.n & 1) == 0 && np >= 2) {   // 16-byte state accesses (row starts stay 16-byte aligned)
        switch (np) {
            SFDA_STEP_PAIR_CASE(2) SFDA_STEP_PAIR_CASE(4) SFDA_STEP_PAIR_CASE(8)
            SFDA_STEP_PAIR_CASE(16) SFDA_STEP_PAIR_CASE(32) SFDA_STEP_PAIR_CASE(64)
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    switch (np) {
        SFDA_STEP_CASE(1) SFDA_STEP_CASE(2) SFDA_STEP_CASE(4) SFDA_STEP_CASE(8)
        SFDA_STEP_CASE(16) SFDA_STEP_CASE(32) SFDA_STEP_CASE(64)
        default: return hipErrorInvalidValue;
    }
#undef SFDA_STEP_CASE
#undef SFDA_STEP_PAIR_CASE
    return hipGetLastError();
}

hipError_t launch_step(const StepLaunch& L, hipStream_t st)
{
    if (L.in_bf16) {
        return L.out_bf16 ? launch_step_t<uint16_t, uint16_t>(L, st) : launch_step_t<uint16_t, float>(L, st);
    }
    return L.out_bf16 ? launch_step_t<float, uint16_t>(L, st) : launch_step_t<float, float>(L, st);
}

}  // namespace sfda
