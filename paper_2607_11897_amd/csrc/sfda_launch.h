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
};

struct GateParams {
    bool gated;
    float alpha_min, alpha_max, theta_max, eps;
};

hipError_t launch_step(const StepLaunch& L, hipStream_t st);
hipError_t launch_chunk(const ChunkLaunch& L, hipStream_t st);
hipError_t launch_chunk_bf16(const ChunkLaunch& L, hipStream_t st);   // bf16 inputs
// segment-parallel scan: identity fill and the fold of the segments' affine maps
hipError_t launch_identity(float* P, long count, int m, hipStream_t st);
hipError_t launch_fold(const float* P, const float* Bs, float* Sin, const float* S0, float* S_T,
                       long heads, int G, int m, int n, hipStream_t st);

}  // namespace sfda
