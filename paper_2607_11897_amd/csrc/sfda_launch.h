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
    const void *q, *k, *v, *alpha, *theta, *beta;
    const float* S0;   // may be null (zero state)
    void* o;
    float* S_T;        // may be null
    int B, H, T, m, n, C;
    int slice;         // value columns per workgroup (multiple of 8, <= 64)
    bool in_bf16, out_bf16;
};

hipError_t launch_step(const StepLaunch& L, hipStream_t st);
hipError_t launch_chunk(const ChunkLaunch& L, hipStream_t st);
hipError_t launch_chunk_bf16(const ChunkLaunch& L, hipStream_t st);   // bf16 inputs

}  // namespace sfda
