// Host-side launch descriptors passed from the C-ABI layer to the kernel launchers.
// Arguments are already validated when these are filled in.
#pragma once

#include <hip/hip_runtime.h>

namespace sfda {

struct StepLaunch {
    const void *q, *k, *v, *alpha, *theta, *beta;
    float* S;
    void* o;
    int B, H, m, n;
    bool in_bf16, out_bf16;
};

struct ChunkLaunch {
    const void *q, *k, *v, *alpha, *theta, *beta;   // v may be null (zero values)
    const float* S0;   // may be null (zero state)
    void* o;           // may be null (no output)
    float* S_T;        // may be null
    int B, H, T, m, n, C;
    int slice;         // value columns per workgroup (multiple of 8, <= 64)
    bool in_bf16, out_bf16;
    // gated: alpha, theta, beta, k hold the pre-activations a, b, c and the raw keys, mapped
    // by alpha = alpha_min + (alpha_max - alpha_min) sigmoid(a), theta = theta_max tanh(b),
    // beta = sigmoid(c), k = k~ / (||k~|| + eps)
    bool gated = false;
    float alpha_min = 0.f, alpha_max = 1.f, theta_max = 0.f, eps = 0.f;
    // backward scans (launch_bwd_scans): per-chunk records
    // [heads][chunks][m][n] and [heads][chunks * C][n] (complex fp32); the adjoint scan
    // reads dL/do (o's dtype) and writes dL/dv (the inputs' dtype), and takes dL/dS_T in
    // S0 and writes dL/dS0 to S_T
    float* ck_state = nullptr;
    float* ck_rows = nullptr;
    const void* dO = nullptr;
    void* dv = nullptr;
    // write-decoupled forward (launch_chunk_decoupled): write directions r and write
    // strengths wbeta; beta holds the erase strengths
    const void* r = nullptr;
    const void* wbeta = nullptr;
    // segment forward (launch_chunk_segment): beside the value columns (from S0 = 0 when
    // S0 is null) the m columns of the homogeneous transfer from I_m, with outputs
    // X_t = P_t^* q_t [heads][T][m] and the last transfer [heads][m][m] (complex fp32)
    float* xo = nullptr;
    float* pend = nullptr;
};

// per-chunk gradient pass of the backward (one workgroup per head and chunk)
struct GradLaunch {
    const void *q, *k, *v, *alpha, *theta, *beta;   // the forward's inputs
    const void* dO;                                 // dL/do, o's dtype
    const float *S_rec, *G_rec;                     // [heads][chunks][m][n]: S entering, dL/dS leaving
    const float *D_rows, *F_rows;                   // [heads][chunks * C][n]: Delta, G_F
    void *dq, *dk, *dalpha, *dtheta, *dbeta;        // the inputs' dtype
    int B, H, T, m, n, C;
    bool in_bf16, out_bf16;
};

// bfloat16 inputs with at most this many key channels take float32 matrix-core operands:
// with one or two channels the erase factor (1 - beta |k|^2) can come close to zero, and the
// cancellation in (I - beta k k^*) S then magnifies the rounding of bf16 operands past the
// bf16 bar (fp32 operands keep it near the fp32 level); at these sizes the cost is nil
constexpr int SMALL_M_FP32_OPERANDS = 4;
inline bool bf16_operands(bool in_bf16, int m) { return in_bf16 && m > SMALL_M_FP32_OPERANDS; }

struct GateParams {
    bool gated;
    float alpha_min, alpha_max, theta_max, eps;
};

hipError_t launch_step(const StepLaunch& L, hipStream_t st);
hipError_t launch_chunk(const ChunkLaunch& L, hipStream_t st);
hipError_t launch_chunk_bf16(const ChunkLaunch& L, hipStream_t st);   // bf16 inputs
hipError_t launch_chunk_decoupled(const ChunkLaunch& L, hipStream_t st);   // C = 16 or 32
hipError_t launch_chunk_segment(const ChunkLaunch& L, hipStream_t st);
// backward: the forward scan recording states and Delta (F; none when F.T == 0) and the
// reverse adjoint scan (A) in one launch, then the per-chunk gradient pass
hipError_t launch_bwd_scans(const ChunkLaunch& F, const ChunkLaunch& A, hipStream_t st);
hipError_t launch_chunk_grad(const GradLaunch& L, hipStream_t st);
// per 16-token block: the triangular solve's residual and ||D_beta L'||_F ([B, H, ceil(T / 16)])
hipError_t launch_solve_monitor(const ChunkLaunch& L, float* residual, float* lnorm, hipStream_t st);
// segment-parallel scan: identity fill, the fold of the segments' affine maps and the join of
// the outputs (o += S_in^* X)
hipError_t launch_identity(float* P, long count, int m, hipStream_t st);
hipError_t launch_join(const float* X, const float* Sin, void* o, bool out_bf16, long segs,
                       int Ts, int m, int n, hipStream_t st);
hipError_t launch_fold(const float* P, const float* Bs, float* Sin, const float* S0, float* S_T,
                       long heads, int G, int m, int n, hipStream_t st);

}  // namespace sfda
