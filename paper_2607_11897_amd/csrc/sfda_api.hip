// C-ABI entry points of libsfda: argument validation, then one kernel launch.
#include <stdint.h>

#include <mutex>

#include "../../include/sfda.h"
#include "sfda_launch.h"

// Workspace of sfda_chunk_fwd_segmented_noalloc: a file-scope device array, one copy per GPU
// the library runs on, held until the process ends.  In host code its name is only a
// stand-in; the device address comes from hipGetSymbolAddress (per device, with that device
// current) and only that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[SFDA_NOALLOC_SCRATCH_BYTES];

namespace {

struct Range {
    uintptr_t lo, hi;   // [lo, hi)
};

Range range_of(const void* p, long bytes) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    return Range{a, a + static_cast<uintptr_t>(bytes > 0 ? bytes : 0)};
}

bool overlap(Range a, Range b) {
    return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

long esize(sfda_dtype_t d) { return d == SFDA_BF16 ? 2 : 4; }

bool dtype_ok(sfda_dtype_t d) { return d == SFDA_F32 || d == SFDA_BF16; }

// the device address of `scratch` on the current device, looked up once per device
constexpr int MAX_DEVICES = 64;
std::mutex scratch_mu;
void* scratch_ptr[MAX_DEVICES];

sfda_status_t scratch_address(void** out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return SFDA_ERR_HIP;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return SFDA_ERR_HIP;
        scratch_ptr[dev] = p;
    }
    *out = scratch_ptr[dev];
    return SFDA_OK;
}

// compute units of the current device (0 if it cannot be queried), looked up once per device
std::mutex cu_mu;
int cu_count_cache[MAX_DEVICES];

int device_cus()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return 0;
    std::lock_guard<std::mutex> lock(cu_mu);
    if (cu_count_cache[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        cu_count_cache[dev] = v;
    }
    return cu_count_cache[dev];
}

// sfda_chunk_fwd's value columns per workgroup: all of a head's columns (up to 64), halved
// to 32 while the heads alone would leave more than half of the compute units idle (each
// workgroup scans its head's sequence on one compute unit; the column slices of a head repeat
// its chunk factors but scan in parallel).  Every column's arithmetic is the same for every
// slice, so the results do not depend on it.
int auto_slice(long BH, int n)
{
    int slice = n <= 64 ? ((n + 7) / 8) * 8 : 64;
    const long cus = device_cus();
    if (slice > 32 && cus > 0 && 2 * BH * ((n + slice - 1) / slice) <= cus) slice = 32;
    return slice;
}

}  // namespace

extern "C" {

const char* sfda_status_string(sfda_status_t s)
{
    switch (s) {
        case SFDA_OK: return "ok";
        case SFDA_ERR_NULL: return "a required pointer is NULL";
        case SFDA_ERR_SHAPE: return "a size is out of range";
        case SFDA_ERR_CHUNK: return "unsupported chunk length (C must be 16, 32, 64 or 128)";
        case SFDA_ERR_DTYPE: return "unsupported dtype";
        case SFDA_ERR_ALIGN: return "a pointer is not 16-byte aligned";
        case SFDA_ERR_ALIAS: return "an output buffer overlaps another buffer";
        case SFDA_ERR_HIP: return "the HIP runtime reported an error";
        case SFDA_ERR_SCRATCH: return "the call needs more workspace than the static scratch holds";
    }
    return "unknown status";
}

int sfda_abi_version(void) { return SFDA_ABI_VERSION; }

// one head's state (m x n complex float32) is addressed with 32-bit byte offsets
static bool state_fits(int m, int n) { return static_cast<long>(m) * n * 8 < 0x80000000L; }
// the float32 path addresses one chunk's rows of v, o and dL/do (C x n complex, at most 8
// bytes per element, C <= 32 in those kernels) with 32-bit byte offsets
static bool chunk_rows_fit(int n) { return static_cast<long>(32) * n * 8 < 0x80000000L; }
// chunk lengths the entry points accept (the kernels' blocking does not change the result,
// Thm 6.1)
static bool chunk_ok(int C) { return C == 16 || C == 32 || C == 64 || C == 128; }

static sfda_status_t chunk_fwd_impl(const void* q, const void* k, const void* v,
                                    const void* alpha, const void* theta, const void* beta,
                                    const float* S0, void* o, float* S_T, int B, int H, int T,
                                    int m, int n, int C, sfda_dtype_t in_dtype,
                                    sfda_dtype_t out_dtype, sfda_stream_t stream, int slice,
                                    void* = nullptr, size_t = 0, bool check_only = false,
                                    const sfda::GateParams* gates = nullptr)
{
    if (!dtype_ok(in_dtype) || !dtype_ok(out_dtype)) return SFDA_ERR_DTYPE;
    if (B < 0 || H < 0 || T < 0 || m < 1 || m > 64 || n < 1 || !state_fits(m, n)) return SFDA_ERR_SHAPE;
    if (!chunk_ok(C)) return SFDA_ERR_CHUNK;
    if (!chunk_rows_fit(n)) return SFDA_ERR_SHAPE;
    if (slice < 8 || slice > 64 || (slice & 7) != 0) return SFDA_ERR_SHAPE;
    const long BH = static_cast<long>(B) * H;
    if (BH * ((n + slice - 1) / slice) > 0x7FFFFFFFL) return SFDA_ERR_SHAPE;
    // bf16 inputs: each head's slice of q, k, v and o is addressed with 32-bit byte offsets
    if (in_dtype == SFDA_BF16 &&
        static_cast<long>(T) * (m > n ? m : n) * 2 * esize(out_dtype) >= 0x80000000L)
        return SFDA_ERR_SHAPE;
    if (BH == 0) return SFDA_OK;
    const bool need_inputs = T > 0;
    if (need_inputs && (!q || !k || !v || !alpha || !theta || !beta || !o)) return SFDA_ERR_NULL;
    const void* ptrs[] = {q, k, v, alpha, theta, beta, S0, o, S_T};
    for (const void* p : ptrs)
        if (p && !aligned16(p)) return SFDA_ERR_ALIGN;

    const long ei = esize(in_dtype), eo = esize(out_dtype);
    const long BHT = BH * T;
    const Range rq = range_of(q, BHT * m * 2 * ei), rk = range_of(k, BHT * m * 2 * ei);
    const Range rv = range_of(v, BHT * n * 2 * ei);
    const Range ra = range_of(alpha, BHT * m * ei), rt = range_of(theta, BHT * m * ei);
    const Range rb = range_of(beta, BHT * ei);
    const Range ro = range_of(o, BHT * n * 2 * eo);
    const Range rs0 = range_of(S0, BH * m * n * 2 * 4);
    const Range rst = range_of(S_T, BH * m * n * 2 * 4);
    const Range ins[] = {rq, rk, rv, ra, rt, rb};
    if (need_inputs) {
        for (const Range& r : ins)
            if (overlap(ro, r)) return SFDA_ERR_ALIAS;
        if (overlap(ro, rs0) || overlap(ro, rst)) return SFDA_ERR_ALIAS;
    }
    if (S_T) {
        if (need_inputs)
            for (const Range& r : ins)
                if (overlap(rst, r)) return SFDA_ERR_ALIAS;
        if (S0 && static_cast<const void*>(S0) != static_cast<const void*>(S_T) && overlap(rs0, rst))
            return SFDA_ERR_ALIAS;
    }

    if (check_only) return SFDA_OK;
    sfda::ChunkLaunch L;
    L.q = q; L.k = k; L.v = v; L.alpha = alpha; L.theta = theta; L.beta = beta;
    L.S0 = S0; L.o = o; L.S_T = S_T;
    L.B = B; L.H = H; L.T = T; L.m = m; L.n = n; L.C = C; L.slice = slice;
    L.in_bf16 = in_dtype == SFDA_BF16;
    L.out_bf16 = out_dtype == SFDA_BF16;
    if (gates) {
        L.gated = gates->gated;
        L.alpha_min = gates->alpha_min; L.alpha_max = gates->alpha_max;
        L.theta_max = gates->theta_max; L.eps = gates->eps;
    }
    const hipError_t e = sfda::launch_chunk(L, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SFDA_OK : SFDA_ERR_HIP;
}

sfda_status_t sfda_chunk_fwd(const void* q, const void* k, const void* v, const void* alpha,
                             const void* theta, const void* beta, const float* S0, void* o,
                             float* S_T, int B, int H, int T, int m, int n, int C,
                             sfda_dtype_t in_dtype, sfda_dtype_t out_dtype, sfda_stream_t stream)
{
    const int slice = auto_slice(static_cast<long>(B) * H, n);
    return chunk_fwd_impl(q, k, v, alpha, theta, beta, S0, o, S_T, B, H, T, m, n, C, in_dtype,
                          out_dtype, stream, slice);
}

sfda_status_t sfda_chunk_fwd_sliced(const void* q, const void* k, const void* v,
                                    const void* alpha, const void* theta, const void* beta,
                                    const float* S0, void* o, float* S_T, int B, int H, int T,
                                    int m, int n, int C, int slice, sfda_dtype_t in_dtype,
                                    sfda_dtype_t out_dtype, sfda_stream_t stream)
{
    return chunk_fwd_impl(q, k, v, alpha, theta, beta, S0, o, S_T, B, H, T, m, n, C, in_dtype,
                          out_dtype, stream, slice);
}

sfda_status_t sfda_chunk_fwd_gated(const void* q, const void* k_raw, const void* v,
                                   const void* a, const void* b, const void* c,
                                   const float* S0, void* o, float* S_T, int B, int H, int T,
                                   int m, int n, int C, float alpha_min, float alpha_max,
                                   float theta_max, float eps, sfda_dtype_t in_dtype,
                                   sfda_dtype_t out_dtype, sfda_stream_t stream)
{
    // ALPHA_MIN_GATED <= alpha_min <= alpha_max <= 1: the kernels' 16-token blocks divide by
    // the decay over one block, which stays inside the float range (>= 2^-126) whenever every
    // alpha is at least 2^(-126/16); theta_max and eps finite and >= 0 (NaN fails every
    // comparison)
    constexpr float ALPHA_MIN_GATED = 0.0042719f;     // 2^(-7.875), rounded up
    if (!(alpha_min >= ALPHA_MIN_GATED && alpha_min <= alpha_max && alpha_max <= 1.f)) return SFDA_ERR_SHAPE;
    if (!(theta_max >= 0.f && theta_max < 3.4e38f && eps >= 0.f && eps < 3.4e38f)) return SFDA_ERR_SHAPE;
    const int slice = auto_slice(static_cast<long>(B) * H, n);
    sfda::GateParams gp{true, alpha_min, alpha_max, theta_max, eps};
    return chunk_fwd_impl(q, k_raw, v, a, b, c, S0, o, S_T, B, H, T, m, n, C, in_dtype, out_dtype,
                          stream, slice, nullptr, 0, false, &gp);
}

sfda_status_t sfda_chunk_fwd_decoupled(const void* q, const void* k, const void* r, const void* v,
                                       const void* alpha, const void* theta, const void* eta,
                                       const void* beta, const float* S0, void* o, float* S_T,
                                       int B, int H, int T, int m, int n, int C,
                                       sfda_dtype_t in_dtype, sfda_dtype_t out_dtype,
                                       sfda_stream_t stream)
{
    const int slice = auto_slice(static_cast<long>(B) * H, n);
    // the shared checks, with the erase strengths in beta's place
    const sfda_status_t st0 = chunk_fwd_impl(q, k, v, alpha, theta, eta, S0, o, S_T, B, H, T, m, n,
                                             C, in_dtype, out_dtype, stream, slice, nullptr, 0,
                                             /*check_only=*/true);
    if (st0 != SFDA_OK) return st0;
    const long BH = static_cast<long>(B) * H;
    if (BH == 0) return SFDA_OK;
    if (T > 0 && (!r || !beta)) return SFDA_ERR_NULL;
    if ((r && !aligned16(r)) || (beta && !aligned16(beta))) return SFDA_ERR_ALIGN;
    const long ei = esize(in_dtype), eo = esize(out_dtype), BHT = BH * T;
    const Range rr = range_of(r, BHT * m * 2 * ei), rb = range_of(beta, BHT * ei);
    if (T > 0 && (overlap(range_of(o, BHT * n * 2 * eo), rr) || overlap(range_of(o, BHT * n * 2 * eo), rb)))
        return SFDA_ERR_ALIAS;
    if (S_T && T > 0 && (overlap(range_of(S_T, BH * m * n * 2 * 4), rr) || overlap(range_of(S_T, BH * m * n * 2 * 4), rb)))
        return SFDA_ERR_ALIAS;
    sfda::ChunkLaunch L;
    L.q = q; L.k = k; L.v = v; L.alpha = alpha; L.theta = theta; L.beta = eta;
    L.r = r; L.wbeta = beta;
    L.S0 = S0; L.o = o; L.S_T = S_T;
    L.B = B; L.H = H; L.T = T; L.m = m; L.n = n; L.C = C; L.slice = slice;
    L.in_bf16 = in_dtype == SFDA_BF16;
    L.out_bf16 = out_dtype == SFDA_BF16;
    const hipError_t e = sfda::launch_chunk_decoupled(L, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SFDA_OK : SFDA_ERR_HIP;
}

size_t sfda_chunk_fwd_segmented_workspace_bytes(int B, int H, int T, int m, int n, int G,
                                                sfda_dtype_t in_dtype)
{
    if (B <= 0 || H <= 0 || T < 0 || m < 1 || m > 64 || n < 1 || G < 1 || !dtype_ok(in_dtype)) return 0;
    const size_t segs = static_cast<size_t>(B) * H * G, heads = static_cast<size_t>(B) * H;
    // per segment P_g (m x m), B_g and S_in (m x n); with float32 inputs per head and token
    // X_t (m)
    const size_t xt = in_dtype == SFDA_F32 ? heads * static_cast<size_t>(T) * m : 0;
    return (segs * (static_cast<size_t>(m) * m + 2 * static_cast<size_t>(m) * n) + xt) * 8;
}

int sfda_chunk_fwd_auto_segments(int B, int H, int T, int m, int n, int C, sfda_dtype_t in_dtype)
{
    if (B <= 0 || H <= 0 || T <= 0 || m < 1 || m > 64 || n < 1 || !chunk_ok(C) || !dtype_ok(in_dtype))
        return 1;
    const long cus = device_cus();
    if (cus <= 0) return 1;
    const long per = static_cast<long>(B) * H * ((n + 63) / 64);     // workgroups per segment index
    int G = 1;
    while (G < 1024 && per * 2 * G <= cus && T % (2L * G * C) == 0 && T / (2L * G) >= 256) G *= 2;
    // the segmented scan repeats the scan work twice (float32) or three times (bfloat16)
    return G >= (in_dtype == SFDA_F32 ? 4 : 8) ? G : 1;
}

// sfda_chunk_fwd_segmented, and with noalloc the workspace taken from the static scratch
// (its size checked first, its address fetched only after every other argument check)
static sfda_status_t segmented_impl(const void* q, const void* k, const void* v,
                                    const void* alpha, const void* theta, const void* beta,
                                    const float* S0, void* o, float* S_T, int B, int H, int T,
                                    int m, int n, int C, int G, sfda_dtype_t in_dtype,
                                    sfda_dtype_t out_dtype, void* workspace,
                                    size_t workspace_bytes, sfda_stream_t stream, bool noalloc)
{
    if (G < 1) return SFDA_ERR_SHAPE;
    const int slice_n = n <= 64 ? ((n + 7) / 8) * 8 : 64;
    // the shared checks (and the whole call when there is nothing to split)
    if (T == 0 || static_cast<long>(B) * H == 0 || !dtype_ok(in_dtype) || !dtype_ok(out_dtype) ||
        B < 0 || H < 0 || T < 0 || m < 1 || m > 64 || n < 1 || !state_fits(m, n) || !chunk_ok(C))
        return chunk_fwd_impl(q, k, v, alpha, theta, beta, S0, o, S_T, B, H, T, m, n, C, in_dtype,
                              out_dtype, stream, slice_n);
    if (T % (static_cast<long>(G) * C) != 0) return SFDA_ERR_SHAPE;
    const long BH = static_cast<long>(B) * H;
    if (BH * G > 0x7FFFFFFFL) return SFDA_ERR_SHAPE;
    if (noalloc) {
        if (sfda_chunk_fwd_segmented_workspace_bytes(B, H, T, m, n, G, in_dtype) > SFDA_NOALLOC_SCRATCH_BYTES)
            return SFDA_ERR_SCRATCH;
        const sfda_status_t st0 = chunk_fwd_impl(q, k, v, alpha, theta, beta, S0, o, S_T, B, H, T,
                                                 m, n, C, in_dtype, out_dtype, stream, slice_n,
                                                 nullptr, 0, /*check_only=*/true);
        if (st0 != SFDA_OK) return st0;
        const sfda_status_t st1 = scratch_address(&workspace);
        if (st1 != SFDA_OK) return st1;
        workspace_bytes = SFDA_NOALLOC_SCRATCH_BYTES;
    }
    if (!workspace) return SFDA_ERR_NULL;
    if (!aligned16(workspace)) return SFDA_ERR_ALIGN;
    const size_t need = sfda_chunk_fwd_segmented_workspace_bytes(B, H, T, m, n, G, in_dtype);
    if (workspace_bytes < need) return SFDA_ERR_SHAPE;
    // validate the buffers the way sfda_chunk_fwd does (nothing is launched on error)
    {
        const sfda_status_t st0 = chunk_fwd_impl(q, k, v, alpha, theta, beta, S0, o, S_T, B, H, T,
                                                 m, n, C, in_dtype, out_dtype, stream, slice_n,
                                                 nullptr, 0, /*check_only=*/true);
        if (st0 != SFDA_OK) return st0;
    }
    const long ei = esize(in_dtype), eo = esize(out_dtype), BHT = BH * T;
    const Range rw = range_of(workspace, static_cast<long>(need));
    const Range all[] = {range_of(q, BHT * m * 2 * ei), range_of(k, BHT * m * 2 * ei),
                         range_of(v, BHT * n * 2 * ei), range_of(alpha, BHT * m * ei),
                         range_of(theta, BHT * m * ei), range_of(beta, BHT * ei),
                         range_of(o, BHT * n * 2 * eo), range_of(S0, BH * m * n * 2 * 4),
                         range_of(S_T, BH * m * n * 2 * 4)};
    for (const Range& r : all)
        if (overlap(rw, r)) return SFDA_ERR_ALIAS;

    const hipStream_t st = static_cast<hipStream_t>(stream);
    const long segs = BH * G;
    float* P = static_cast<float*>(workspace);                      // [segs][m][m]
    float* Bs = P + segs * m * m * 2;                               // [segs][m][n]
    float* Sin = Bs + segs * static_cast<long>(m) * n * 2;          // [segs][m][n]
    float* X = Sin + segs * static_cast<long>(m) * n * 2;           // [segs][T / G][m], float32 inputs
    // [B, H, T, .] with T = G * Ts is [B*H*G, Ts, .]: each segment runs as a head
    const int Ts = T / G;
    // float32 inputs: the outputs come from the zero-state pass and a join (o0 + S_in^* X),
    // cheaper than a third pass of the latency-bound float32 scan; bfloat16 inputs: a third
    // pass of the pipelined kernel from the incoming states (cheaper than writing X in
    // float32 and the join)
    const bool join = in_dtype == SFDA_F32 && o != nullptr;
    sfda::ChunkLaunch L;
    L.q = q; L.k = k; L.alpha = alpha; L.theta = theta; L.beta = beta;
    L.B = static_cast<int>(segs); L.H = 1; L.T = Ts; L.m = m; L.C = C;
    L.in_bf16 = in_dtype == SFDA_BF16;
    if (join && n <= 64) {
        // P_g and B_g in one scan per segment (one copy of the chunk factors): the transfer
        // columns from I_m with X_t = P_t^* q_t, the value columns from zero with o0 into o
        L.v = v; L.S0 = nullptr; L.S_T = Bs; L.o = o; L.out_bf16 = out_dtype == SFDA_BF16;
        L.n = n; L.slice = slice_n; L.xo = X; L.pend = P;
        if (sfda::launch_chunk_segment(L, st) != hipSuccess) return SFDA_ERR_HIP;
    } else {
        // P_g (and with the join X_t = P_t^* q_t, the m-column float32 output): S0 = I,
        // v = 0, in place on the identity
        if (sfda::launch_identity(P, segs, m, st) != hipSuccess) return SFDA_ERR_HIP;
        L.v = nullptr; L.S0 = P; L.S_T = P; L.o = join ? X : nullptr; L.out_bf16 = false;
        L.n = m; L.slice = ((m + 7) / 8) * 8;
        if (sfda::launch_chunk(L, st) != hipSuccess) return SFDA_ERR_HIP;
        // B_g (and with the join the zero-state outputs o0, into o)
        L.v = v; L.S0 = nullptr; L.S_T = Bs; L.o = join ? o : nullptr; L.out_bf16 = out_dtype == SFDA_BF16;
        L.n = n; L.slice = slice_n;
        if (sfda::launch_chunk(L, st) != hipSuccess) return SFDA_ERR_HIP;
    }
    // incoming states and S_T
    if (sfda::launch_fold(P, Bs, Sin, S0, S_T, BH, G, m, n, st) != hipSuccess) return SFDA_ERR_HIP;
    if (join) {
        // o = o0 + S_in^* X (the affine law of each segment, token by token)
        if (sfda::launch_join(X, Sin, o, out_dtype == SFDA_BF16, segs, Ts, m, n, st) != hipSuccess)
            return SFDA_ERR_HIP;
    } else {
        // outputs from the exact incoming states
        L.S0 = Sin; L.S_T = nullptr; L.o = o;
        if (sfda::launch_chunk(L, st) != hipSuccess) return SFDA_ERR_HIP;
    }
    return SFDA_OK;
}

sfda_status_t sfda_chunk_fwd_segmented(const void* q, const void* k, const void* v,
                                       const void* alpha, const void* theta, const void* beta,
                                       const float* S0, void* o, float* S_T, int B, int H, int T,
                                       int m, int n, int C, int G, sfda_dtype_t in_dtype,
                                       sfda_dtype_t out_dtype, void* workspace,
                                       size_t workspace_bytes, sfda_stream_t stream)
{
    return segmented_impl(q, k, v, alpha, theta, beta, S0, o, S_T, B, H, T, m, n, C, G, in_dtype,
                          out_dtype, workspace, workspace_bytes, stream, false);
}

sfda_status_t sfda_chunk_fwd_segmented_noalloc(const void* q, const void* k, const void* v,
                                               const void* alpha, const void* theta,
                                               const void* beta, const float* S0, void* o,
                                               float* S_T, int B, int H, int T, int m, int n,
                                               int C, int G, sfda_dtype_t in_dtype,
                                               sfda_dtype_t out_dtype, sfda_stream_t stream)
{
    return segmented_impl(q, k, v, alpha, theta, beta, S0, o, S_T, B, H, T, m, n, C, G, in_dtype,
                          out_dtype, nullptr, 0, stream, true);
}

// the backward's chunk length: C = 64 and 128 run at 32 (the gradient pass stages a block
// of value columns beside the chunk's operands in LDS; every C gives the same gradients up
// to rounding)
// The backward runs 16-token chunks whatever C is (the gradients do not depend on the
// chunk length, to rounding): 1 / g of a 16-token chunk stays finite while the chunk's
// decay is at least 2^-126, the forward's range, and measured on MI355X it is as fast as
// 32-token chunks (the scans' steps are shorter, the gradient pass has twice the
// workgroups).
static int bwd_chunk(int) { return 16; }

size_t sfda_chunk_bwd_workspace_bytes(int B, int H, int T, int m, int n, int C)
{
    if (B <= 0 || H <= 0 || T < 0 || m < 1 || m > 64 || n < 1) return 0;
    if (!chunk_ok(C)) return 0;
    C = bwd_chunk(C);
    const size_t chunks = static_cast<size_t>(B) * H * ((static_cast<size_t>(T) + C - 1) / C);
    // per chunk: S entering and dL/dS leaving (m x n each), Delta and G_F (C x n each)
    return chunks * (2 * static_cast<size_t>(m) * n + 2 * static_cast<size_t>(C) * n) * 8;
}

sfda_status_t sfda_chunk_bwd(const void* q, const void* k, const void* v, const void* alpha,
                             const void* theta, const void* beta, const float* S0,
                             const void* dO, const float* dS_T, void* dq, void* dk, void* dv,
                             void* dalpha, void* dtheta, void* dbeta, float* dS0, int B, int H,
                             int T, int m, int n, int C, sfda_dtype_t in_dtype,
                             sfda_dtype_t out_dtype, void* workspace, size_t workspace_bytes,
                             sfda_stream_t stream)
{
    if (!dtype_ok(in_dtype) || !dtype_ok(out_dtype)) return SFDA_ERR_DTYPE;
    if (B < 0 || H < 0 || T < 0 || m < 1 || m > 64 || n < 1 || !state_fits(m, n)) return SFDA_ERR_SHAPE;
    if (!chunk_ok(C)) return SFDA_ERR_CHUNK;
    if (!chunk_rows_fit(n)) return SFDA_ERR_SHAPE;
    const size_t need = sfda_chunk_bwd_workspace_bytes(B, H, T, m, n, C);
    C = bwd_chunk(C);
    const long BH = static_cast<long>(B) * H;
    const int slice = n <= 64 ? ((n + 7) / 8) * 8 : 64;
    const long nchunks = (static_cast<long>(T) + C - 1) / C;
    if (BH * ((n + slice - 1) / slice) > 0x7FFFFFFFL || BH * nchunks > 0x7FFFFFFFL) return SFDA_ERR_SHAPE;
    if (BH == 0) return SFDA_OK;
    const bool need_inputs = T > 0;
    if (need_inputs && (!q || !k || !v || !alpha || !theta || !beta || !dO || !dq || !dk || !dv ||
                        !dalpha || !dtheta || !dbeta))
        return SFDA_ERR_NULL;
    if (need > 0 && !workspace) return SFDA_ERR_NULL;
    const void* ptrs[] = {q, k, v, alpha, theta, beta, S0, dO, dS_T, dq, dk, dv, dalpha, dtheta,
                          dbeta, dS0, workspace};
    for (const void* p : ptrs)
        if (p && !aligned16(p)) return SFDA_ERR_ALIGN;
    if (workspace_bytes < need) return SFDA_ERR_SHAPE;

    const long ei = esize(in_dtype), eo = esize(out_dtype), BHT = BH * T;
    const Range ins[] = {range_of(q, BHT * m * 2 * ei), range_of(k, BHT * m * 2 * ei),
                         range_of(v, BHT * n * 2 * ei), range_of(alpha, BHT * m * ei),
                         range_of(theta, BHT * m * ei), range_of(beta, BHT * ei),
                         range_of(S0, BH * m * n * 2 * 4), range_of(dO, BHT * n * 2 * eo),
                         range_of(dS_T, BH * m * n * 2 * 4)};
    const Range outs[] = {range_of(dq, BHT * m * 2 * ei), range_of(dk, BHT * m * 2 * ei),
                          range_of(dv, BHT * n * 2 * ei), range_of(dalpha, BHT * m * ei),
                          range_of(dtheta, BHT * m * ei), range_of(dbeta, BHT * ei),
                          range_of(dS0, BH * m * n * 2 * 4),
                          range_of(workspace, static_cast<long>(need))};
    for (int a = 0; a < 8; ++a) {
        for (const Range& r : ins)
            if (overlap(outs[a], r)) return SFDA_ERR_ALIAS;
        for (int b = a + 1; b < 8; ++b)
            if (overlap(outs[a], outs[b])) return SFDA_ERR_ALIAS;
    }

    const hipStream_t st = static_cast<hipStream_t>(stream);
    float* S_rec = static_cast<float*>(workspace);
    float* G_rec = S_rec + BH * nchunks * m * n * 2;
    float* D_rows = G_rec + BH * nchunks * m * n * 2;
    float* F_rows = D_rows + BH * nchunks * C * n * 2;
    sfda::ChunkLaunch L;
    L.q = q; L.k = k; L.v = v; L.alpha = alpha; L.theta = theta; L.beta = beta;
    L.B = B; L.H = H; L.T = T; L.m = m; L.n = n; L.C = C; L.slice = slice;
    L.in_bf16 = in_dtype == SFDA_BF16;
    L.out_bf16 = out_dtype == SFDA_BF16;
    L.o = nullptr;
    // forward scan (the state entering every chunk and Delta) and reverse scan (dL/dS leaving
    // every chunk, G_F, dv and dS0; with T == 0 only dS0 = dS_T), in one launch
    sfda::ChunkLaunch F = L;
    F.S0 = S0; F.S_T = nullptr; F.ck_state = S_rec; F.ck_rows = D_rows;
    L.S0 = dS_T; L.S_T = dS0; L.ck_state = G_rec; L.ck_rows = F_rows; L.dO = dO; L.dv = dv;
    if (sfda::launch_bwd_scans(F, L, st) != hipSuccess) return SFDA_ERR_HIP;
    if (!need_inputs) return SFDA_OK;
    sfda::GradLaunch Gl;
    Gl.q = q; Gl.k = k; Gl.v = v; Gl.alpha = alpha; Gl.theta = theta; Gl.beta = beta; Gl.dO = dO;
    Gl.S_rec = S_rec; Gl.G_rec = G_rec; Gl.D_rows = D_rows; Gl.F_rows = F_rows;
    Gl.dq = dq; Gl.dk = dk; Gl.dalpha = dalpha; Gl.dtheta = dtheta; Gl.dbeta = dbeta;
    Gl.B = B; Gl.H = H; Gl.T = T; Gl.m = m; Gl.n = n; Gl.C = C;
    Gl.in_bf16 = L.in_bf16; Gl.out_bf16 = L.out_bf16;
    if (sfda::launch_chunk_grad(Gl, st) != hipSuccess) return SFDA_ERR_HIP;
    return SFDA_OK;
}

sfda_status_t sfda_chunk_solve_monitor(const void* k, const void* alpha, const void* theta,
                                       const void* beta, float* residual, float* lnorm, int B,
                                       int H, int T, int m, sfda_dtype_t in_dtype,
                                       sfda_stream_t stream)
{
    if (!dtype_ok(in_dtype)) return SFDA_ERR_DTYPE;
    if (B < 0 || H < 0 || T < 0 || m < 1 || m > 64) return SFDA_ERR_SHAPE;
    const long BH = static_cast<long>(B) * H, nb = (static_cast<long>(T) + 15) / 16;
    if (BH * nb > 0x7FFFFFFFL) return SFDA_ERR_SHAPE;
    if (BH == 0 || T == 0) return SFDA_OK;
    if (!k || !alpha || !theta || !beta || (!residual && !lnorm)) return SFDA_ERR_NULL;
    const void* ptrs[] = {k, alpha, theta, beta, residual, lnorm};
    for (const void* p : ptrs)
        if (p && !aligned16(p)) return SFDA_ERR_ALIGN;
    const long ei = esize(in_dtype), BHT = BH * T;
    const Range ins[] = {range_of(k, BHT * m * 2 * ei), range_of(alpha, BHT * m * ei),
                         range_of(theta, BHT * m * ei), range_of(beta, BHT * ei)};
    const Range outs[] = {range_of(residual, BH * nb * 4), range_of(lnorm, BH * nb * 4)};
    for (const Range& o : outs)
        for (const Range& r : ins)
            if (overlap(o, r)) return SFDA_ERR_ALIAS;
    if (overlap(outs[0], outs[1])) return SFDA_ERR_ALIAS;
    sfda::ChunkLaunch L;
    L.q = k; L.k = k; L.v = nullptr; L.alpha = alpha; L.theta = theta; L.beta = beta;
    L.S0 = nullptr; L.o = nullptr; L.S_T = nullptr;
    L.B = B; L.H = H; L.T = T; L.m = m; L.n = 8; L.C = 16; L.slice = 8;
    L.in_bf16 = in_dtype == SFDA_BF16;
    L.out_bf16 = false;
    if (sfda::launch_solve_monitor(L, residual, lnorm, static_cast<hipStream_t>(stream)) != hipSuccess)
        return SFDA_ERR_HIP;
    return SFDA_OK;
}

sfda_status_t sfda_step(const void* q, const void* k, const void* v, const void* alpha,
                        const void* theta, const void* beta, float* S, void* o, int B, int H,
                        int m, int n, sfda_dtype_t in_dtype, sfda_dtype_t out_dtype,
                        sfda_stream_t stream)
{
    if (!dtype_ok(in_dtype) || !dtype_ok(out_dtype)) return SFDA_ERR_DTYPE;
    if (B < 0 || H < 0 || m < 1 || m > 64 || n < 1 || !state_fits(m, n)) return SFDA_ERR_SHAPE;
    if (n >= (1 << 22)) return SFDA_ERR_SHAPE;   // state rows addressed with 32-bit offsets
    const long BH = static_cast<long>(B) * H;
    int np = 1;
    while (np < n && np < 64) np <<= 1;
    if (BH * ((n + np - 1) / np) > 0x7FFFFFFFL) return SFDA_ERR_SHAPE;
    if (BH == 0) return SFDA_OK;
    if (!q || !k || !v || !alpha || !theta || !beta || !S || !o) return SFDA_ERR_NULL;
    const void* ptrs[] = {q, k, v, alpha, theta, beta, S, o};
    for (const void* p : ptrs)
        if (!aligned16(p)) return SFDA_ERR_ALIGN;
    const long ei = esize(in_dtype), eo = esize(out_dtype);
    const Range ins[] = {range_of(q, BH * m * 2 * ei), range_of(k, BH * m * 2 * ei),
                         range_of(v, BH * n * 2 * ei), range_of(alpha, BH * m * ei),
                         range_of(theta, BH * m * ei), range_of(beta, BH * ei)};
    const Range rs = range_of(S, BH * m * n * 2 * 4);
    const Range ro = range_of(o, BH * n * 2 * eo);
    if (overlap(ro, rs)) return SFDA_ERR_ALIAS;
    for (const Range& r : ins)
        if (overlap(ro, r) || overlap(rs, r)) return SFDA_ERR_ALIAS;

    sfda::StepLaunch L;
    L.q = q; L.k = k; L.v = v; L.alpha = alpha; L.theta = theta; L.beta = beta;
    L.S = S; L.o = o; L.B = B; L.H = H; L.m = m; L.n = n;
    L.in_bf16 = in_dtype == SFDA_BF16;
    L.out_bf16 = out_dtype == SFDA_BF16;
    const hipError_t e = sfda::launch_step(L, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SFDA_OK : SFDA_ERR_HIP;
}

}  // extern "C"
