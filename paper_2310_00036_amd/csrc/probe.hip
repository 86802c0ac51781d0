// Achievable matrix-core throughput on this device: a loop of independent
// v_mfma_f32_16x16x32_bf16 on operands held in registers (no memory traffic inside the loop),
// the ceiling a kernel's MFMA work can reach here, measured beside the published dense peak.
// The loop is written as inline assembly: compiled from the builtin, the loop-carried
// accumulators are copied between register files every round, which would understate the
// ceiling. The s_nop padding covers the wait states around the asm block that the compiler's
// hazard checks do not see (operands written by VALU before it, results read by VALU after).
#include "common.h"
#include "kernels.h"

namespace cb {

constexpr int kProbeChains = 8;   // independent accumulators per wave

__global__ __launch_bounds__(256) void mfma_probe_kernel(float* sink, int iters) {
    const uint32_t lane = threadIdx.x & 63u;
    // finite bf16 operands that differ per lane
    const uint32_t av = pack2bf(1.f + float(lane) / 128.f, 1.f);
    const uint32_t bv = pack2bf(1.f - float(lane) / 256.f, 0.5f);
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 a = {av, av, av, av}, b = {bv, bv, bv, bv};
    cb_f32x4 c0{}, c1{}, c2{}, c3{}, c4{}, c5{}, c6{}, c7{};
    // the nops take the operands, so they follow the instructions that write them
    asm volatile("s_nop 7\n\ts_nop 7" : "+v"(c0), "+v"(c1), "+v"(c2), "+v"(c3), "+v"(c4), "+v"(c5), "+v"(c6), "+v"(c7)
                 : "v"(a), "v"(b));
    for (int i = 0; i < iters; ++i) {
        asm volatile(
            "v_mfma_f32_16x16x32_bf16 %0, %8, %9, %0\n\t"
            "v_mfma_f32_16x16x32_bf16 %1, %8, %9, %1\n\t"
            "v_mfma_f32_16x16x32_bf16 %2, %8, %9, %2\n\t"
            "v_mfma_f32_16x16x32_bf16 %3, %8, %9, %3\n\t"
            "v_mfma_f32_16x16x32_bf16 %4, %8, %9, %4\n\t"
            "v_mfma_f32_16x16x32_bf16 %5, %8, %9, %5\n\t"
            "v_mfma_f32_16x16x32_bf16 %6, %8, %9, %6\n\t"
            "v_mfma_f32_16x16x32_bf16 %7, %8, %9, %7"
            : "+v"(c0), "+v"(c1), "+v"(c2), "+v"(c3), "+v"(c4), "+v"(c5), "+v"(c6), "+v"(c7)
            : "v"(a), "v"(b));
    }
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+v"(c0), "+v"(c1), "+v"(c2), "+v"(c3), "+v"(c4), "+v"(c5), "+v"(c6), "+v"(c7));
    const cb_f32x4 acc[kProbeChains] = {c0, c1, c2, c3, c4, c5, c6, c7};
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < kProbeChains; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
    sink[int64_t(blockIdx.x) * 256 + threadIdx.x] = s;
}

hipError_t mfma_probe(int blocks, int iters, float* sink, hipStream_t s) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, sink, iters);
    return hipGetLastError();
}

int64_t mfma_probe_flop(int blocks, int iters) {
    return int64_t(blocks) * 4 * iters * kProbeChains * (16 * 16 * 32 * 2);
}

}  // namespace cb
