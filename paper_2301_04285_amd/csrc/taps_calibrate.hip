// taps_calibrate.hip -- measured VALU issue ceilings of the GPU (measurement
// support for the benchmark's roofline, not part of the cost-table path).
//
// Each kernel runs 8 independent dependency chains of one 32-bit integer
// VALU instruction per thread, 8 wavefronts per SIMD (the most a SIMD holds;
// the edge kernel runs 7, as many as its scalar registers allow, and held to
// 8 it ran no faster), so the issue rate, not the latency, bounds it.  The instruction
// count per launch is exact (inline assembly, 16 instructions per block); the
// caller divides it by the measured time.
//   kind 0: v_add_u32 / v_xor_b32 with vector operands -- on gfx950 the class
//           of simple 32-bit operations issued at the highest rate
//   kind 1: v_bfe_u32 / v_lshl_or_b32 -- the class of 3-operand and bit-field
//           operations, issued at a lower rate
//   kinds 2-12: one instruction each (the classes the edge kernels' choice of
//           instructions rests on), 8 per block: see kKindNames
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "taps_calibrate.h"

namespace {

constexpr uint32_t kChains = 8, kSteps = 8;   // instructions per loop iteration: 2 * 8 * 8

__global__ __launch_bounds__(256) void k_valu_fast(uint32_t *out, uint32_t iters, uint32_t c) {
    uint32_t a[kChains];
#pragma unroll
    for (uint32_t k = 0; k < kChains; ++k) a[k] = threadIdx.x * 3u + k + c;
    for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
        for (uint32_t r = 0; r < kSteps; ++r) {
                // 16 instructions in one block: no s_nop between them
                __asm__ volatile(
                    "v_add_u32 %0, %0, %1\n"
                    "v_xor_b32 %0, %0, %3\n"
                    "v_add_u32 %1, %1, %2\n"
                    "v_xor_b32 %1, %1, %4\n"
                    "v_add_u32 %2, %2, %3\n"
                    "v_xor_b32 %2, %2, %5\n"
                    "v_add_u32 %3, %3, %4\n"
                    "v_xor_b32 %3, %3, %6\n"
                    "v_add_u32 %4, %4, %5\n"
                    "v_xor_b32 %4, %4, %7\n"
                    "v_add_u32 %5, %5, %6\n"
                    "v_xor_b32 %5, %5, %0\n"
                    "v_add_u32 %6, %6, %7\n"
                    "v_xor_b32 %6, %6, %1\n"
                    "v_add_u32 %7, %7, %0\n"
                    "v_xor_b32 %7, %7, %2\n"
                    : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(a[4]), "+v"(a[5]),
                      "+v"(a[6]), "+v"(a[7]));
        }
    }
    uint32_t f = 0;
#pragma unroll
    for (uint32_t k = 0; k < kChains; ++k) f ^= a[k];
    out[blockIdx.x * blockDim.x + threadIdx.x] = f;
}

__global__ __launch_bounds__(256) void k_valu_slow(uint32_t *out, uint32_t iters, uint32_t c) {
    uint32_t a[kChains];
#pragma unroll
    for (uint32_t k = 0; k < kChains; ++k) a[k] = threadIdx.x * 3u + k + c;
    for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
        for (uint32_t r = 0; r < kSteps; ++r) {
                // 16 instructions in one block: no s_nop between them
                __asm__ volatile(
                    "v_bfe_u32 %0, %0, %1, 4\n"
                    "v_lshl_or_b32 %0, %0, %2, %3\n"
                    "v_bfe_u32 %1, %1, %2, 4\n"
                    "v_lshl_or_b32 %1, %1, %3, %4\n"
                    "v_bfe_u32 %2, %2, %3, 4\n"
                    "v_lshl_or_b32 %2, %2, %4, %5\n"
                    "v_bfe_u32 %3, %3, %4, 4\n"
                    "v_lshl_or_b32 %3, %3, %5, %6\n"
                    "v_bfe_u32 %4, %4, %5, 4\n"
                    "v_lshl_or_b32 %4, %4, %6, %7\n"
                    "v_bfe_u32 %5, %5, %6, 4\n"
                    "v_lshl_or_b32 %5, %5, %7, %0\n"
                    "v_bfe_u32 %6, %6, %7, 4\n"
                    "v_lshl_or_b32 %6, %6, %0, %1\n"
                    "v_bfe_u32 %7, %7, %0, 4\n"
                    "v_lshl_or_b32 %7, %7, %1, %2\n"
                    : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(a[4]), "+v"(a[5]),
                      "+v"(a[6]), "+v"(a[7]));
        }
    }
    uint32_t f = 0;
#pragma unroll
    for (uint32_t k = 0; k < kChains; ++k) f ^= a[k];
    out[blockIdx.x * blockDim.x + threadIdx.x] = f;
}

// One instruction per chain step, 16 per block as in the kernels above: chain
// k takes operands from chains k+1 and k+2 (vector registers) or from a scalar
// register c.
#define TAPS_CAL_KERNEL(NAME, I0, I1, I2, I3, I4, I5, I6, I7)                                    \
    __global__ __launch_bounds__(256) void NAME(uint32_t *out, uint32_t iters, uint32_t c) {      \
        uint32_t a[kChains];                                                                   \
        _Pragma("unroll") for (uint32_t k = 0; k < kChains; ++k) a[k] = threadIdx.x * 3u + k + c; \
        for (uint32_t i = 0; i < iters; ++i) {                                                 \
            _Pragma("unroll") for (uint32_t r = 0; r < kSteps; ++r) {                           \
                __asm__ volatile(I0 "\n" I1 "\n" I2 "\n" I3 "\n" I4 "\n" I5 "\n" I6 "\n" I7  \
                                 "\n" I0 "\n" I1 "\n" I2 "\n" I3 "\n" I4 "\n" I5 "\n" I6     \
                                 "\n" I7                                                       \
                                 : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(a[4]),   \
                                   "+v"(a[5]), "+v"(a[6]), "+v"(a[7])                         \
                                 : "s"(c));                                                    \
            }                                                                                  \
        }                                                                                      \
        uint32_t f = 0;                                                                        \
        _Pragma("unroll") for (uint32_t k = 0; k < kChains; ++k) f ^= a[k];                    \
        out[blockIdx.x * blockDim.x + threadIdx.x] = f;                                        \
    }

// expands the operand pattern into the kernel's 8 instruction arguments
#define TAPS_CAL_KERNEL_(...) TAPS_CAL_KERNEL(__VA_ARGS__)

// operand patterns: two vector sources (chains k+1, k+2), or a scalar one (%8)
#define TAPS_CAL_V2(OP)                                                                          \
    OP " %0, %1, %2", OP " %1, %2, %3", OP " %2, %3, %4", OP " %3, %4, %5", OP " %4, %5, %6",    \
        OP " %5, %6, %7", OP " %6, %7, %0", OP " %7, %0, %1"
#define TAPS_CAL_V3(OP, SUF)                                                                     \
    OP " %0, %0, %1, %2" SUF, OP " %1, %1, %2, %3" SUF, OP " %2, %2, %3, %4" SUF,                \
        OP " %3, %3, %4, %5" SUF, OP " %4, %4, %5, %6" SUF, OP " %5, %5, %6, %7" SUF,            \
        OP " %6, %6, %7, %0" SUF, OP " %7, %7, %0, %1" SUF
#define TAPS_CAL_S(OP)                                                                           \
    OP " %0, %8, %0", OP " %1, %8, %1", OP " %2, %8, %2", OP " %3, %8, %3", OP " %4, %8, %4",    \
        OP " %5, %8, %5", OP " %6, %8, %6", OP " %7, %8, %7"

TAPS_CAL_KERNEL_(k_cal_bitop3, TAPS_CAL_V3("v_bitop3_b32", " bitop3:0x96"))
TAPS_CAL_KERNEL_(k_cal_and_or, TAPS_CAL_V3("v_and_or_b32", ""))
TAPS_CAL_KERNEL_(k_cal_or3, TAPS_CAL_V3("v_or3_b32", ""))
TAPS_CAL_KERNEL_(k_cal_lshl16, TAPS_CAL_V2("v_lshlrev_b16"))
TAPS_CAL_KERNEL_(k_cal_lshl32, TAPS_CAL_V2("v_lshlrev_b32"))
TAPS_CAL_KERNEL_(k_cal_lshr32, TAPS_CAL_V2("v_lshrrev_b32"))
TAPS_CAL_KERNEL_(k_cal_bcnt, TAPS_CAL_V2("v_bcnt_u32_b32"))
TAPS_CAL_KERNEL_(k_cal_bfm, TAPS_CAL_V2("v_bfm_b32"))
TAPS_CAL_KERNEL_(k_cal_and, TAPS_CAL_V2("v_and_b32"))
TAPS_CAL_KERNEL_(k_cal_and_s, TAPS_CAL_S("v_and_b32"))
TAPS_CAL_KERNEL_(k_cal_add_s, TAPS_CAL_S("v_add_u32"))

using cal_kernel = void (*)(uint32_t *, uint32_t, uint32_t);
// kinds 2 .. 12
const cal_kernel kKinds[] = {k_cal_bitop3, k_cal_and_or, k_cal_or3,  k_cal_lshl16,
                             k_cal_lshl32, k_cal_lshr32, k_cal_bcnt, k_cal_bfm,
                             k_cal_and,    k_cal_and_s,  k_cal_add_s};
const char *const kKindNames[] = {
    "v_add_u32 / v_xor_b32",  "v_bfe_u32 / v_lshl_or_b32", "v_bitop3_b32",
    "v_and_or_b32",           "v_or3_b32",                 "v_lshlrev_b16",
    "v_lshlrev_b32",          "v_lshrrev_b32",             "v_bcnt_u32_b32",
    "v_bfm_b32",              "v_and_b32",                 "v_and_b32, scalar operand",
    "v_add_u32, scalar operand"};
constexpr int kNumKinds = (int)(sizeof(kKindNames) / sizeof(kKindNames[0]));
static_assert(kNumKinds == 2 + (int)(sizeof(kKinds) / sizeof(kKinds[0])), "kind tables");

}  // namespace

extern "C" int taps_calibrate_valu_kinds(void) { return kNumKinds; }

extern "C" const char *taps_calibrate_valu_name(int kind) {
    return kind >= 0 && kind < kNumKinds ? kKindNames[kind] : nullptr;
}

extern "C" int taps_calibrate_valu(int kind, uint32_t iters, float *ms, double *wave_instructions,
                                   uint32_t *simds) {
    if (kind < 0 || kind >= kNumKinds || iters == 0 || !ms || !wave_instructions || !simds) return 1;
    int dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess)
        return 2;
    // 8 blocks of 4 wavefronts per CU: 8 wavefronts on each of its 4 SIMDs
    const uint32_t blocks = (uint32_t)prop.multiProcessorCount * 8u;
    uint32_t *out = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int rc = 0;
    if (hipMalloc(&out, (size_t)blocks * 256u * sizeof(uint32_t)) != hipSuccess) return 3;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) rc = 4;
    float best = 0.f;
    for (int rep = 0; rc == 0 && rep < 3; ++rep) {
        (void)hipEventRecord(e0, nullptr);
        if (kind == 0)
            hipLaunchKernelGGL(k_valu_fast, dim3(blocks), dim3(256), 0, nullptr, out, iters, 7u);
        else if (kind == 1)
            hipLaunchKernelGGL(k_valu_slow, dim3(blocks), dim3(256), 0, nullptr, out, iters, 7u);
        else
            hipLaunchKernelGGL(kKinds[kind - 2], dim3(blocks), dim3(256), 0, nullptr, out, iters, 7u);
        if (hipGetLastError() != hipSuccess) rc = 5;
        (void)hipEventRecord(e1, nullptr);
        float t = 0.f;
        if (rc == 0 && (hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(&t, e0, e1) != hipSuccess))
            rc = 6;
        if (rc == 0 && (rep == 0 || t < best)) best = t;
    }
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    (void)hipFree(out);
    if (rc) return rc;
    *ms = best;
    *wave_instructions = (double)blocks * 4.0 * iters * 2.0 * kSteps * kChains;
    *simds = (uint32_t)prop.multiProcessorCount * 4u;
    return 0;
}
