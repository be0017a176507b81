// Measurement aid for the instruction-issue rooflines: the rate at which the
// chip retires wave-wide 32-bit integer VALU instructions when nothing else
// competes (no memory traffic, no scalar work inside the timed loop, eight
// independent dependency chains per lane, every wave slot filled), and the
// shader clock the chip ran at meanwhile.  The nominal figure the rooflines
// use is one such instruction per CU per clock.
#include "pc_internal.h"

#include <type_traits>

namespace {

constexpr int kPeakThreads = 256;
constexpr int kPeakPerIter = 64;  // instructions per loop iteration: 8 on each of 8 chains

// Op 0: v_add_u32 / v_sub_u32 (VOP2); 1: v_xor_b32 (VOP2); 2: v_and_or_b32
// with three vector sources (VOP3); 3: v_and_or_b32 with two vector sources
// and one scalar (VOP3); 4: v_lshlrev_b64 by a scalar amount (VOP3, 64-bit);
// 5: v_add_u32 in its VOP3 encoding; 6: s_xor_b32 on scalar registers (the
// scalar ALU, one chain set per wavefront); 7: v_mov_b64 (each move reads the
// previous one's destination); 8: v_cmp_ne_u32 into scalar register pairs;
// 9: v_cndmask_b32 selecting by a scalar register pair; 10: v_bfi_b32 (three
// vector sources); 11: v_xor_b32 with one scalar source; 12: v_mov_b32
// (VOP1, each reading the previous one's destination); 13: v_xor_b32 with an
// inline constant; 14: v_xor_b32 with a 32-bit literal.  The values do not matter, only that each instruction
// depends on the previous one of its chain.
template <int Op>
__global__ __launch_bounds__(kPeakThreads) void k_valu_peak(int32_t iters, uint32_t seed, uint32_t *sink,
                                                            uint64_t *clk)
{
    using T = std::conditional_t<Op == 4 || Op == 7, uint64_t, uint32_t>;
    T a0 = (Op == 6 ? 0u : threadIdx.x) ^ seed, a1 = a0 + 1u, a2 = a0 + 2u, a3 = a0 + 3u;
    T a4 = a0 + 4u, a5 = a0 + 5u, a6 = a0 + 6u, a7 = a0 + 7u;
    const uint32_t k = seed | 1u, m = seed >> 3;
    // the first wavefront of the first workgroup reads the shader-clock and
    // constant-rate counters around its loop, while the whole chip is loaded
    const bool probe = clk != nullptr && blockIdx.x == 0 && threadIdx.x < 64;
    uint64_t t0 = 0, w0 = 0;
    if (probe) {
        t0 = __builtin_amdgcn_s_memtime();
        w0 = __builtin_amdgcn_s_memrealtime();
    }
#define PC_R2(op)                                                                              \
    "v_" op " %0, %0, %8\n\tv_" op " %1, %1, %8\n\tv_" op " %2, %2, %8\n\tv_" op " %3, %3, %8\n\t" \
    "v_" op " %4, %4, %8\n\tv_" op " %5, %5, %8\n\tv_" op " %6, %6, %8\n\tv_" op " %7, %7, %8\n\t"
#define PC_R3(op)                                                                                        \
    "v_" op " %0, %0, %8, %9\n\tv_" op " %1, %1, %8, %9\n\tv_" op " %2, %2, %8, %9\n\tv_" op " %3, %3, %8, %9\n\t" \
    "v_" op " %4, %4, %8, %9\n\tv_" op " %5, %5, %8, %9\n\tv_" op " %6, %6, %8, %9\n\tv_" op " %7, %7, %8, %9\n\t"
#define PC_SH                                                                                      \
    "v_lshlrev_b64 %0, %8, %0\n\tv_lshlrev_b64 %1, %8, %1\n\tv_lshlrev_b64 %2, %8, %2\n\t"          \
    "v_lshlrev_b64 %3, %8, %3\n\tv_lshlrev_b64 %4, %8, %4\n\tv_lshlrev_b64 %5, %8, %5\n\t"          \
    "v_lshlrev_b64 %6, %8, %6\n\tv_lshlrev_b64 %7, %8, %7\n\t"
#define PC_S2                                                                                     \
    "s_xor_b32 %0, %0, %8\n\ts_xor_b32 %1, %1, %8\n\ts_xor_b32 %2, %2, %8\n\ts_xor_b32 %3, %3, %8\n\t"  \
    "s_xor_b32 %4, %4, %8\n\ts_xor_b32 %5, %5, %8\n\ts_xor_b32 %6, %6, %8\n\ts_xor_b32 %7, %7, %8\n\t"
// moves rotate the eight 64-bit values so each reads the last one written
#define PC_MV                                                                                     \
    "v_mov_b64 %0, %7\n\tv_mov_b64 %1, %0\n\tv_mov_b64 %2, %1\n\tv_mov_b64 %3, %2\n\t"               \
    "v_mov_b64 %4, %3\n\tv_mov_b64 %5, %4\n\tv_mov_b64 %6, %5\n\tv_mov_b64 %7, %6\n\t"
#define PC_CMP                                                                                    \
    "v_cmp_ne_u32_e64 %0, %8, %16\n\tv_cmp_ne_u32_e64 %1, %9, %16\n\tv_cmp_ne_u32_e64 %2, %10, %16\n\t"  \
    "v_cmp_ne_u32_e64 %3, %11, %16\n\tv_cmp_ne_u32_e64 %4, %12, %16\n\tv_cmp_ne_u32_e64 %5, %13, %16\n\t" \
    "v_cmp_ne_u32_e64 %6, %14, %16\n\tv_cmp_ne_u32_e64 %7, %15, %16\n\t"
#define PC_CND                                                                                    \
    "v_cndmask_b32_e64 %0, %0, %8, %9\n\tv_cndmask_b32_e64 %1, %1, %8, %9\n\t"                          \
    "v_cndmask_b32_e64 %2, %2, %8, %9\n\tv_cndmask_b32_e64 %3, %3, %8, %9\n\t"                          \
    "v_cndmask_b32_e64 %4, %4, %8, %9\n\tv_cndmask_b32_e64 %5, %5, %8, %9\n\t"                          \
    "v_cndmask_b32_e64 %6, %6, %8, %9\n\tv_cndmask_b32_e64 %7, %7, %8, %9\n\t"
#define PC_R2S                                                                                    \
    "v_xor_b32 %0, %8, %0\n\tv_xor_b32 %1, %8, %1\n\tv_xor_b32 %2, %8, %2\n\tv_xor_b32 %3, %8, %3\n\t"  \
    "v_xor_b32 %4, %8, %4\n\tv_xor_b32 %5, %8, %5\n\tv_xor_b32 %6, %8, %6\n\tv_xor_b32 %7, %8, %7\n\t"
#define PC_MV32                                                                                   \
    "v_mov_b32 %0, %7\n\tv_mov_b32 %1, %0\n\tv_mov_b32 %2, %1\n\tv_mov_b32 %3, %2\n\t"               \
    "v_mov_b32 %4, %3\n\tv_mov_b32 %5, %4\n\tv_mov_b32 %6, %5\n\tv_mov_b32 %7, %6\n\t"
#define PC_RC(c)                                                                                  \
    "v_xor_b32 %0, " c ", %0\n\tv_xor_b32 %1, " c ", %1\n\tv_xor_b32 %2, " c ", %2\n\t"                   \
    "v_xor_b32 %3, " c ", %3\n\tv_xor_b32 %4, " c ", %4\n\tv_xor_b32 %5, " c ", %5\n\t"                   \
    "v_xor_b32 %6, " c ", %6\n\tv_xor_b32 %7, " c ", %7\n\t"
    for (int32_t i = 0; i < iters; ++i) {
        if constexpr (Op == 0) {
            asm volatile(PC_R2("add_u32") PC_R2("sub_u32") PC_R2("add_u32") PC_R2("sub_u32")
                         PC_R2("add_u32") PC_R2("sub_u32") PC_R2("add_u32") PC_R2("sub_u32")
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "v"(k), "v"(m));
        } else if constexpr (Op == 1) {
            asm volatile(PC_R2("xor_b32") PC_R2("xor_b32") PC_R2("xor_b32") PC_R2("xor_b32")
                         PC_R2("xor_b32") PC_R2("xor_b32") PC_R2("xor_b32") PC_R2("xor_b32")
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "v"(k), "v"(m));
        } else if constexpr (Op == 2) {
            asm volatile(PC_R3("and_or_b32") PC_R3("and_or_b32") PC_R3("and_or_b32") PC_R3("and_or_b32")
                         PC_R3("and_or_b32") PC_R3("and_or_b32") PC_R3("and_or_b32") PC_R3("and_or_b32")
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "v"(k), "v"(m));
        } else if constexpr (Op == 3) {
            asm volatile(PC_R3("and_or_b32") PC_R3("and_or_b32") PC_R3("and_or_b32") PC_R3("and_or_b32")
                         PC_R3("and_or_b32") PC_R3("and_or_b32") PC_R3("and_or_b32") PC_R3("and_or_b32")
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "v"(k), "s"(m));
        } else if constexpr (Op == 5) {
            asm volatile(PC_R2("add_u32_e64") PC_R2("sub_u32_e64") PC_R2("add_u32_e64") PC_R2("sub_u32_e64")
                         PC_R2("add_u32_e64") PC_R2("sub_u32_e64") PC_R2("add_u32_e64") PC_R2("sub_u32_e64")
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "v"(k), "v"(m));
        } else if constexpr (Op == 6) {
            asm volatile(PC_S2 PC_S2 PC_S2 PC_S2 PC_S2 PC_S2 PC_S2 PC_S2
                         : "+s"(a0), "+s"(a1), "+s"(a2), "+s"(a3), "+s"(a4), "+s"(a5), "+s"(a6), "+s"(a7)
                         : "s"(k)
                         : "scc");  // s_xor_b32 writes the scalar condition code
        } else if constexpr (Op == 7) {
            asm volatile(PC_MV PC_MV PC_MV PC_MV PC_MV PC_MV PC_MV PC_MV
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7));
        } else if constexpr (Op == 8) {
            uint64_t c0, c1, c2, c3, c4, c5, c6, c7;
            asm volatile(PC_CMP PC_CMP PC_CMP PC_CMP PC_CMP PC_CMP PC_CMP PC_CMP
                         : "=s"(c0), "=s"(c1), "=s"(c2), "=s"(c3), "=s"(c4), "=s"(c5), "=s"(c6), "=s"(c7)
                         : "v"(a0), "v"(a1), "v"(a2), "v"(a3), "v"(a4), "v"(a5), "v"(a6), "v"(a7), "v"(k));
            a0 ^= static_cast<uint32_t>(c0 ^ c1 ^ c2 ^ c3 ^ c4 ^ c5 ^ c6 ^ c7);
        } else if constexpr (Op == 9) {
            const uint64_t sel = (static_cast<uint64_t>(seed) << 32) | (seed * 2654435761u);
            asm volatile(PC_CND PC_CND PC_CND PC_CND PC_CND PC_CND PC_CND PC_CND
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "v"(k), "s"(sel));
        } else if constexpr (Op == 10) {
            asm volatile(PC_R3("bfi_b32") PC_R3("bfi_b32") PC_R3("bfi_b32") PC_R3("bfi_b32")
                         PC_R3("bfi_b32") PC_R3("bfi_b32") PC_R3("bfi_b32") PC_R3("bfi_b32")
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "v"(k), "v"(m));
        } else if constexpr (Op == 11) {
            asm volatile(PC_R2S PC_R2S PC_R2S PC_R2S PC_R2S PC_R2S PC_R2S PC_R2S
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "s"(k));
        } else if constexpr (Op == 12) {
            asm volatile(PC_MV32 PC_MV32 PC_MV32 PC_MV32 PC_MV32 PC_MV32 PC_MV32 PC_MV32
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7));
        } else if constexpr (Op == 13) {
            asm volatile(PC_RC("15") PC_RC("15") PC_RC("15") PC_RC("15") PC_RC("15") PC_RC("15") PC_RC("15")
                         PC_RC("15")
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7));
        } else if constexpr (Op == 14) {
            asm volatile(PC_RC("0x5bd1e995") PC_RC("0x5bd1e995") PC_RC("0x5bd1e995") PC_RC("0x5bd1e995")
                         PC_RC("0x5bd1e995") PC_RC("0x5bd1e995") PC_RC("0x5bd1e995") PC_RC("0x5bd1e995")
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7));
        } else {
            asm volatile(PC_SH PC_SH PC_SH PC_SH PC_SH PC_SH PC_SH PC_SH
                         : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3), "+v"(a4), "+v"(a5), "+v"(a6), "+v"(a7)
                         : "s"(k));
        }
    }
#undef PC_R2
#undef PC_R3
#undef PC_SH
#undef PC_S2
#undef PC_MV
#undef PC_CMP
#undef PC_CND
#undef PC_R2S
#undef PC_MV32
#undef PC_RC
    if (probe) {
        const uint64_t t1 = __builtin_amdgcn_s_memtime();
        const uint64_t w1 = __builtin_amdgcn_s_memrealtime();
        if (threadIdx.x == 0) {
            clk[0] = t1 - t0;
            clk[1] = w1 - w0;
        }
    }
    // keeps the chains live; never fires for a seed below 2^31
    if (static_cast<uint32_t>(a0 ^ a1 ^ a2 ^ a3 ^ a4 ^ a5 ^ a6 ^ a7) == 0xFFFFFFFFu && (seed >> 31))
        sink[threadIdx.x] = static_cast<uint32_t>(a0);
}

}  // namespace

extern "C" int pc_measure_valu(pc_ctx *ctx, int op, int reps, double *wave_instr_per_s, double *clock_hz,
                               void *stream_)
{
    if (!ctx || !wave_instr_per_s || reps < 1 || op < 0 || op > 14) return PC_EINVAL;
    hipStream_t stream = static_cast<hipStream_t>(stream_);
    PC_HIP(ctx, hipSetDevice(ctx->device));
    hipDeviceProp_t prop{};
    PC_HIP(ctx, hipGetDeviceProperties(&prop, ctx->device));
    int wall_khz = 0;
    PC_HIP(ctx, hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, ctx->device));
    // every wave slot: 8 workgroups of 4 wavefronts per CU (32 waves), 4 rounds
    const unsigned grid = static_cast<unsigned>(prop.multiProcessorCount) * 8u * 4u;
    const int32_t iters = 2048;
    using Kern = void (*)(int32_t, uint32_t, uint32_t *, uint64_t *);
    static const Kern kernels[] = {k_valu_peak<0>, k_valu_peak<1>, k_valu_peak<2>, k_valu_peak<3>,
                                   k_valu_peak<4>, k_valu_peak<5>, k_valu_peak<6>, k_valu_peak<7>,
                                   k_valu_peak<8>, k_valu_peak<9>, k_valu_peak<10>, k_valu_peak<11>,
                                   k_valu_peak<12>, k_valu_peak<13>, k_valu_peak<14>};
    const Kern kern = kernels[op];
    uint64_t *d_clk = nullptr;
    if (clock_hz) PC_HIP(ctx, hipMalloc(&d_clk, 2 * sizeof(uint64_t)));
    hipEvent_t e0, e1;
    PC_HIP(ctx, hipEventCreate(&e0));
    PC_HIP(ctx, hipEventCreate(&e1));
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kPeakThreads), 0, stream, iters, 12345u, nullptr, nullptr);
    PC_LAUNCH_CHECK(ctx);
    PC_HIP(ctx, hipEventRecord(e0, stream));
    for (int r = 0; r < reps; ++r)
        hipLaunchKernelGGL(kern, dim3(grid), dim3(kPeakThreads), 0, stream, iters, 12345u, nullptr,
                           r == reps - 1 ? d_clk : nullptr);
    PC_LAUNCH_CHECK(ctx);
    PC_HIP(ctx, hipEventRecord(e1, stream));
    PC_HIP(ctx, hipEventSynchronize(e1));
    float ms = 0.f;
    PC_HIP(ctx, hipEventElapsedTime(&ms, e0, e1));
    PC_HIP(ctx, hipEventDestroy(e0));
    PC_HIP(ctx, hipEventDestroy(e1));
    const double waves = static_cast<double>(grid) * (kPeakThreads / 64);
    const double instr = waves * iters * static_cast<double>(kPeakPerIter) * reps;
    *wave_instr_per_s = ms > 0.f ? instr / (ms * 1e-3) : 0.0;
    if (clock_hz) {
        uint64_t h[2] = {0, 0};
        PC_HIP(ctx, hipMemcpy(h, d_clk, sizeof(h), hipMemcpyDeviceToHost));
        PC_HIP(ctx, hipFree(d_clk));
        // shader cycles over the constant-rate counter's seconds
        *clock_hz = (h[1] > 0 && wall_khz > 0) ? static_cast<double>(h[0]) / (h[1] / (wall_khz * 1e3)) : 0.0;
    }
    return PC_OK;
}
