// Machine microbenchmarks (gfx950): bf16 matrix-core rate, v_exp_f32 rate,
// the two in one instruction stream, streaming HBM reads and writes, and the
// shader clock under load. They set the ceilings the DAR kernels are measured
// against: the distant region of the prefill issues one exponential per
// score (Eq. 4's softmax) for only 4 * d_down matrix flops, and the decode
// reads the split cache once per step.
//
// Every kernel writes at most: one fp32 to sink[0] (under a data-dependent
// condition that does not hold, so the work cannot be removed), four 64-bit
// clock stamps (first wavefront of workgroup 0), and, for the write stream,
// the caller's buffer within its size.
#include <hip/hip_runtime.h>

#include "../../include/dar_k0.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;  // 4 wavefronts: one per SIMD of a compute unit

__device__ __forceinline__ void stamp(unsigned long long* clk, int at) {
    if (__builtin_amdgcn_workgroup_id_x() == 0 && __builtin_amdgcn_workitem_id_x() == 0) {
        clk[at] = __builtin_amdgcn_s_memtime();          // shader clock cycles
        clk[at + 1] = __builtin_amdgcn_s_memrealtime();  // 100 MHz constant clock
    }
}

__device__ __forceinline__ bf16x8_t operand(float base) {
    bf16x8_t r;
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = (__bf16)(base + 0.001f * j);
    return r;
}

// NM matrix ops and NE vector ops per loop iteration, on 4 independent
// accumulators and 16 independent chains per lane. OP selects the vector op:
// 0 v_exp_f32, 1 v_fma_f32.
template <int NM, int NE, int OP = 0>
__global__ __launch_bounds__(kThreads) void k0_pipes(float* sink, unsigned long long* clk, int iters,
                                                     float seed) {
    stamp(clk, 0);
    const float lane = (float)(__builtin_amdgcn_workitem_id_x() & 63);
    const bf16x8_t a = operand(seed * 1e-3f + lane * 1e-5f);
    const bf16x8_t b = operand(seed * 2e-3f);
    f32x16_t acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
    float x[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) x[j] = 0.25f + 0.01f * j + lane * 1e-4f * seed;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int m = 0; m < NM; ++m)
            acc[m & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[m & 3], 0, 0, 0);
        // x = 2^-x keeps every chain inside [0.5, 1]: one v_exp_f32 each
        // (the negation is a source modifier)
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            if (OP == 0) {
                x[e & 15] = __builtin_amdgcn_exp2f(-x[e & 15]);
            } else {
                x[e & 15] = __builtin_fmaf(x[e & 15], 0.999f, 0.0005f);
            }
        }
    }
    float s = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[t][r];
#pragma unroll
    for (int j = 0; j < 16; ++j) s += x[j];
    stamp(clk, 2);
    if (s == -1.2345f) sink[0] = s;
}

__global__ __launch_bounds__(kThreads) void k0_read(const uint4* __restrict__ p, size_t n, float* sink) {
    const size_t stride = (size_t)__builtin_amdgcn_grid_size_x();  // threads in the grid
    uint32_t acc = 0;
    for (size_t i = (size_t)__builtin_amdgcn_workgroup_id_x() * kThreads + __builtin_amdgcn_workitem_id_x();
         i < n; i += stride) {
        const uint4 v = p[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9e3779b9u) sink[0] = (float)acc;
}

__global__ __launch_bounds__(kThreads) void k0_write(uint4* __restrict__ p, size_t n) {
    const size_t stride = (size_t)__builtin_amdgcn_grid_size_x();
    const uint4 z = make_uint4(0, 0, 0, 0);
    for (size_t i = (size_t)__builtin_amdgcn_workgroup_id_x() * kThreads + __builtin_amdgcn_workitem_id_x();
         i < n; i += stride)
        p[i] = z;
}

struct Timer {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    bool ok = false;
    Timer() { ok = hipEventCreate(&e0) == hipSuccess && hipEventCreate(&e1) == hipSuccess; }
    ~Timer() {
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
    }
};

// Mean time (ms) of `reps` launches after one untimed launch; -1 on error.
template <typename F>
double time_ms(Timer& t, hipStream_t st, int reps, F launch) {
    launch();
    if (hipGetLastError() != hipSuccess || hipStreamSynchronize(st) != hipSuccess) return -1;
    if (hipEventRecord(t.e0, st) != hipSuccess) return -1;
    for (int r = 0; r < reps; ++r) launch();
    if (hipEventRecord(t.e1, st) != hipSuccess) return -1;
    if (hipGetLastError() != hipSuccess || hipEventSynchronize(t.e1) != hipSuccess) return -1;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.e0, t.e1) != hipSuccess) return -1;
    return ms / reps;
}

// Shader clock (MHz) from the stamps of the last launch.
double clock_mhz(unsigned long long* clk_dev, hipStream_t st) {
    unsigned long long h[4] = {0, 0, 0, 0};
    if (hipMemcpyAsync(h, clk_dev, sizeof(h), hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    const double cyc = (double)(h[2] - h[0]), ref = (double)(h[3] - h[1]);
    return ref > 0 ? cyc / ref * 100.0 : -1;
}

}  // namespace

extern "C" int dar_k0_measure(void* buf, size_t buf_bytes, dar_k0_result* out, hipStream_t st) {
    if (!buf || !out || ((uintptr_t)buf & 15u) || buf_bytes < ((size_t)1 << 30)) return 1;
    int dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess) return 5;
    const int n_cu = prop.multiProcessorCount;
    out->n_cu = n_cu;
    Timer tm;
    if (!tm.ok) return 5;
    // the first 256 bytes of buf: sink and clock stamps
    float* sink = (float*)buf;
    unsigned long long* clk = (unsigned long long*)((char*)buf + 64);

    // bf16 matrix-core rate: 4 independent accumulators per wavefront
    const int mfma_iters = 4000;
    const int wps_list[3] = {1, 2, 4};
    for (int c = 0; c < 3; ++c) {
        const int wps = wps_list[c];
        const double ms = time_ms(tm, st, 3, [&] {
            hipLaunchKernelGGL((k0_pipes<4, 0>), dim3(n_cu * wps), dim3(kThreads), 0, st, sink, clk,
                               mfma_iters, 1.f);
        });
        if (ms <= 0) return 5;
        const double flop = (double)n_cu * wps * 4 /* waves */ * mfma_iters * 4 * 32.0 * 32 * 16 * 2;
        out->mfma_bf16_tflops[c] = flop / (ms * 1e-3) / 1e12;
        if (wps == 2) out->mfma_clock_mhz = clock_mhz(clk, st);
    }

    // v_exp_f32 rate, 2 waves per SIMD, 16 chains per lane
    const int exp_iters = 20000;
    {
        const double ms = time_ms(tm, st, 3, [&] {
            hipLaunchKernelGGL((k0_pipes<0, 16>), dim3(n_cu * 2), dim3(kThreads), 0, st, sink, clk,
                               exp_iters, 1.f);
        });
        if (ms <= 0) return 5;
        const double mhz = clock_mhz(clk, st);
        const double lanes = (double)n_cu * 2 * kThreads * exp_iters * 16;
        out->exp_per_s = lanes / (ms * 1e-3);
        out->exp_clock_mhz = mhz;
        out->exp_lanes_per_clk_cu = out->exp_per_s / (mhz * 1e6) / n_cu;
    }

    // 8 matrix ops + 16 exponentials per iteration in one stream, and each
    // part alone; SIMD cycles per wave-iteration at 2 waves per SIMD
    const int mix_iters = 6000;
    double cyc[3];
    for (int c = 0; c < 3; ++c) {
        const double ms = time_ms(tm, st, 3, [&] {
            if (c == 0)
                hipLaunchKernelGGL((k0_pipes<8, 16>), dim3(n_cu * 2), dim3(kThreads), 0, st, sink, clk,
                                   mix_iters, 1.f);
            else if (c == 1)
                hipLaunchKernelGGL((k0_pipes<8, 0>), dim3(n_cu * 2), dim3(kThreads), 0, st, sink, clk,
                                   mix_iters, 1.f);
            else
                hipLaunchKernelGGL((k0_pipes<0, 16>), dim3(n_cu * 2), dim3(kThreads), 0, st, sink, clk,
                                   mix_iters, 1.f);
        });
        if (ms <= 0) return 5;
        const double mhz = clock_mhz(clk, st);
        // each SIMD runs 2 wavefronts of mix_iters iterations
        cyc[c] = ms * 1e-3 * mhz * 1e6 / (2.0 * mix_iters);
    }
    // the same with plain fp32 FMAs instead of exponentials
    double cf[2];
    for (int c = 0; c < 2; ++c) {
        const double ms = time_ms(tm, st, 3, [&] {
            if (c == 0)
                hipLaunchKernelGGL((k0_pipes<0, 16, 1>), dim3(n_cu * 2), dim3(kThreads), 0, st, sink,
                                   clk, mix_iters, 1.f);
            else
                hipLaunchKernelGGL((k0_pipes<8, 16, 1>), dim3(n_cu * 2), dim3(kThreads), 0, st, sink,
                                   clk, mix_iters, 1.f);
        });
        if (ms <= 0) return 5;
        cf[c] = ms * 1e-3 * clock_mhz(clk, st) * 1e6 / (2.0 * mix_iters);
    }
    out->fma_only_cycles_per_iter = cf[0];
    out->mix_fma_cycles_per_iter = cf[1];
    out->mix_cycles_per_iter = cyc[0];
    out->mfma_only_cycles_per_iter = cyc[1];
    out->exp_only_cycles_per_iter = cyc[2];

    // streaming HBM: 16-byte loads / stores, grid-stride, past the first 4 KiB
    const size_t off = 4096;
    const size_t n16 = ((buf_bytes - off) / 16) & ~(size_t)0xffff;
    const uint4* rd = (const uint4*)((const char*)buf + off);
    uint4* wr = (uint4*)((char*)buf + off);
    const double bytes = (double)n16 * 16;
    double best_r = 0, best_w = 0;
    const int bpc_list[3] = {4, 8, 16};
    for (int c = 0; c < 3; ++c) {
        const int blocks = n_cu * bpc_list[c];
        const double mw = time_ms(tm, st, 3, [&] {
            hipLaunchKernelGGL(k0_write, dim3(blocks), dim3(kThreads), 0, st, wr, n16);
        });
        const double mr = time_ms(tm, st, 3, [&] {
            hipLaunchKernelGGL(k0_read, dim3(blocks), dim3(kThreads), 0, st, rd, n16, sink);
        });
        if (mw <= 0 || mr <= 0) return 5;
        const double gw = bytes / (mw * 1e-3) / 1e9, gr = bytes / (mr * 1e-3) / 1e9;
        if (gw > best_w) best_w = gw;
        if (gr > best_r) best_r = gr;
    }
    out->hbm_read_gbs = best_r;
    out->hbm_write_gbs = best_w;
    return 0;
}
