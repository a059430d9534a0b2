// Intra-CU throughput probes for gfx950: the CDNA4 counterpart of the paper's
// rho (APEX4 Sec. 2.2, Eqs. T and rho; Table 1), i.e. the matrix-core integer
// rate over the vector fp32 rate inside one compute unit.  The clock cancels
// in rho, so every probe counts shader-clock cycles (s_memtime) inside the
// kernel instead of wall time.
//
// One workgroup per CU (the dynamic LDS request keeps a second one out), four
// waves per workgroup, so each wave owns one SIMD unless a probe says otherwise.
// Every probe is a bounded loop over registers (or LDS inside the workgroup's
// own allocation); results are written once per wave.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

constexpr int ITERS = 2048;

__device__ __forceinline__ uint64_t cyc() { return __builtin_amdgcn_s_memtime(); }
__device__ __forceinline__ uint64_t rt100() { return __builtin_amdgcn_s_memrealtime(); }

// v_mfma_i32_32x32x32_i8, 4 independent accumulator chains; `vfma` independent
// v_fma_f32 per MFMA interleaved in the same wave.
template <int VFMA, int NT = 256>
__global__ __launch_bounds__(NT) void mfma32_kernel(int seed, uint64_t* cycles, int* sink) {
    i32x4 a = {seed, seed + 1, seed + 2, seed + 3};
    i32x4 b = {seed * 3, seed ^ 5, seed + 7, seed - 1};
    i32x16 acc0 = {}, acc1 = {}, acc2 = {}, acc3 = {};
    float f[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) f[i] = seed * 0.25f + i;
    const float m = 1.0001f, c = 0.5f;
    __builtin_amdgcn_s_barrier();
    const uint64_t t0 = cyc();
    for (int it = 0; it < ITERS; ++it) {
        acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc0, 0, 0, 0);
        if constexpr (VFMA > 0) {
#pragma unroll
            for (int i = 0; i < VFMA; ++i) f[i % 16] = fmaf(f[i % 16], m, c);
        }
        acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc1, 0, 0, 0);
        if constexpr (VFMA > 0) {
#pragma unroll
            for (int i = 0; i < VFMA; ++i) f[(i + 4) % 16] = fmaf(f[(i + 4) % 16], m, c);
        }
        acc2 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc2, 0, 0, 0);
        if constexpr (VFMA > 0) {
#pragma unroll
            for (int i = 0; i < VFMA; ++i) f[(i + 8) % 16] = fmaf(f[(i + 8) % 16], m, c);
        }
        acc3 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc3, 0, 0, 0);
        if constexpr (VFMA > 0) {
#pragma unroll
            for (int i = 0; i < VFMA; ++i) f[(i + 12) % 16] = fmaf(f[(i + 12) % 16], m, c);
        }
        if constexpr (VFMA > 0) {
            // keep one MFMA and VFMA v_fma_f32 together in the schedule
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, VFMA, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, VFMA, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, VFMA, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, VFMA, 0);
        }
    }
    const uint64_t t1 = cyc();
    int s = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc0[i] + acc1[i] + acc2[i] + acc3[i] + static_cast<int>(f[i]);
    if (s == 0x7fffffff) sink[threadIdx.x & 255] = s;
    if ((threadIdx.x & 63) == 0) cycles[blockIdx.x * (NT / 64) + (threadIdx.x >> 6)] = t1 - t0;
}

__global__ __launch_bounds__(256) void mfma16_kernel(int seed, uint64_t* cycles, int* sink) {
    i32x4 a = {seed, seed + 1, seed + 2, seed + 3};
    i32x4 b = {seed * 3, seed ^ 5, seed + 7, seed - 1};
    i32x4 acc[8] = {};
    const uint64_t t0 = cyc();
    for (int it = 0; it < ITERS; ++it) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc[j], 0, 0, 0);
    }
    const uint64_t t1 = cyc();
    int s = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
    if (s == 0x7fffffff) sink[threadIdx.x] = s;
    if ((threadIdx.x & 63) == 0) cycles[blockIdx.x * 4 + (threadIdx.x >> 6)] = t1 - t0;
}

// 16 independent chains of v_fma_f32 (per iteration 16 instructions).
template <int NT = 256>
__global__ __launch_bounds__(NT) void fma_kernel(int seed, uint64_t* cycles, int* sink) {
    float f[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) f[i] = seed * 0.5f + i;
    const float m = 1.0001f, c = 0.5f;
    __builtin_amdgcn_s_barrier();
    const uint64_t t0 = cyc();
    for (int it = 0; it < ITERS; ++it) {
#pragma unroll
        for (int i = 0; i < 16; ++i) f[i] = fmaf(f[i], m, c);
    }
    const uint64_t t1 = cyc();
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += f[i];
    if (s == 1234.5f) sink[threadIdx.x & 255] = 1;
    if ((threadIdx.x & 63) == 0) cycles[blockIdx.x * (NT / 64) + (threadIdx.x >> 6)] = t1 - t0;
}

// 16 independent v_cvt_f32_i32 + v_cvt_i32_f32 pairs per iteration (32 instructions).
__global__ __launch_bounds__(256) void cvt_kernel(int seed, uint64_t* cycles, int* sink) {
    int v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = seed + i;
    const uint64_t t0 = cyc();
    for (int it = 0; it < ITERS; ++it) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            float f = static_cast<float>(v[i]);
            v[i] = static_cast<int>(f) + 1;
        }
    }
    const uint64_t t1 = cyc();
    int s = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += v[i];
    if (s == 0x7fffffff) sink[threadIdx.x] = s;
    if ((threadIdx.x & 63) == 0) cycles[blockIdx.x * 4 + (threadIdx.x >> 6)] = t1 - t0;
}

// Two waves per SIMD (512 threads): waves 0-3 run the MFMA loop, waves 4-7 the
// v_fma_f32 loop; each records its own cycles.
__global__ __launch_bounds__(512) void split_kernel(int seed, uint64_t* cycles, int* sink) {
    const int wave = threadIdx.x >> 6;
    uint64_t t0, t1;
    int s = 0;
    if (wave < 4) {
        i32x4 a = {seed, seed + 1, seed + 2, seed + 3};
        i32x4 b = {seed * 3, seed ^ 5, seed + 7, seed - 1};
        i32x16 acc0 = {}, acc1 = {}, acc2 = {}, acc3 = {};
        t0 = cyc();
        for (int it = 0; it < ITERS; ++it) {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc1, 0, 0, 0);
            acc2 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc2, 0, 0, 0);
            acc3 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc3, 0, 0, 0);
        }
        t1 = cyc();
#pragma unroll
        for (int i = 0; i < 16; ++i) s += acc0[i] + acc1[i] + acc2[i] + acc3[i];
    } else {
        float f[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) f[i] = seed * 0.5f + i;
        const float m = 1.0001f, c = 0.5f;
        t0 = cyc();
        for (int it = 0; it < 2 * ITERS; ++it) {
#pragma unroll
            for (int i = 0; i < 16; ++i) f[i] = fmaf(f[i], m, c);
        }
        t1 = cyc();
#pragma unroll
        for (int i = 0; i < 16; ++i) s += static_cast<int>(f[i]);
    }
    if (s == 0x7fffffff) sink[threadIdx.x] = s;
    if ((threadIdx.x & 63) == 0) cycles[blockIdx.x * 8 + wave] = t1 - t0;
}

// LDS read bandwidth: each lane reads 16 B per ds_read_b128 from a 64 KiB
// window of the workgroup's own dynamic LDS, addresses conflict-free.
__global__ __launch_bounds__(256) void lds_kernel(int seed, uint64_t* cycles, int* sink) {
    extern __shared__ __align__(16) uint8_t lds[];
    uint4* l4 = reinterpret_cast<uint4*>(lds);
    for (int i = threadIdx.x; i < 4096; i += 256) l4[i] = make_uint4(i, seed, i ^ seed, 1);
    __syncthreads();
    uint4 acc = make_uint4(0, 0, 0, 0);
    int idx = threadIdx.x;
    const uint64_t t0 = cyc();
    for (int it = 0; it < ITERS; ++it) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint4 v = l4[(idx + j * 256) & 4095];
            acc.x ^= v.x; acc.y += v.y; acc.z ^= v.z; acc.w += v.w;
        }
        idx = (idx + 64) & 4095;
    }
    const uint64_t t1 = cyc();
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x7fffffffu) sink[threadIdx.x] = 1;
    if ((threadIdx.x & 63) == 0) cycles[blockIdx.x * 4 + (threadIdx.x >> 6)] = t1 - t0;
}


// NCH independent accumulator chains of back-to-back dependent MFMAs.
template <int NCH>
__global__ __launch_bounds__(512) void mfma_chain_kernel(int seed, uint64_t* cycles, int* sink) {
    i32x4 a = {seed, seed + 1, seed + 2, seed + 3};
    i32x4 b = {seed * 3, seed ^ 5, seed + 7, seed - 1};
    i32x16 acc[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) acc[c] = i32x16{};
    const uint64_t t0 = cyc();
    for (int it = 0; it < ITERS; ++it) {
#pragma unroll
        for (int c = 0; c < NCH; ++c) acc[c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[c], 0, 0, 0);
    }
    const uint64_t t1 = cyc();
    int s = 0;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int i = 0; i < 16; ++i) s += acc[c][i];
    if (s == 0x7fffffff) sink[threadIdx.x & 255] = s;
    if ((threadIdx.x & 63) == 0) cycles[blockIdx.x * 8 + (threadIdx.x >> 6)] = t1 - t0;
}

// LDS read bandwidth with WAVES waves per CU and 16 ds_read_b128 in flight per wave.
template <int WAVES>
__global__ __launch_bounds__(64 * WAVES) void lds16_kernel(int seed, uint64_t* cycles, int* sink) {
    extern __shared__ __align__(16) uint8_t lds[];
    uint4* l4 = reinterpret_cast<uint4*>(lds);
    for (int i = threadIdx.x; i < 4096; i += 64 * WAVES) l4[i] = make_uint4(i, seed, i ^ seed, 1);
    __syncthreads();
    uint4 acc = make_uint4(0, 0, 0, 0);
    int idx = threadIdx.x & 255;
    const uint64_t t0 = cyc();
    for (int it = 0; it < ITERS / 2; ++it) {
        uint4 v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = l4[(idx + j * 256) & 4095];
#pragma unroll
        for (int j = 0; j < 16; ++j) { acc.x ^= v[j].x; acc.y += v[j].y; acc.z ^= v[j].z; acc.w += v[j].w; }
        idx = (idx + 64) & 4095;
    }
    const uint64_t t1 = cyc();
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x7fffffffu) sink[threadIdx.x & 255] = 1;
    if ((threadIdx.x & 63) == 0) cycles[blockIdx.x * 8 + (threadIdx.x >> 6)] = t1 - t0;
}

// Shader clock against the 100 MHz constant counter, for a clock estimate.
__global__ void clock_kernel(uint64_t* out) {
    const uint64_t c0 = cyc(), r0 = rt100();
    float f = out[0];
    for (int i = 0; i < 200000; ++i) f = fmaf(f, 1.0000001f, 0.5f);
    const uint64_t c1 = cyc(), r1 = rt100();
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        out[1] = c1 - c0;
        out[2] = r1 - r0;
        out[3] = static_cast<uint64_t>(f);
    }
}

// Plain 16-byte copy: the reference kernel of known traffic that scales the
// FETCH_SIZE / WRITE_SIZE counters to bytes.
__global__ __launch_bounds__(256) void copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

// Plain streaming read (four 16-byte loads in flight per thread): the speed a
// kernel that only reads the same bytes reaches, the practical ceiling for the
// memory-bound GEMMs.  The xor of the data is stored only if it equals a magic
// value, so the loads cannot be dropped.
__global__ __launch_bounds__(256) void read_kernel(const uint4* __restrict__ src, int64_t n, uint32_t* __restrict__ sink) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    uint32_t x = 0;
    for (; i + 3 * stride < n; i += 4 * stride) {
        const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        x ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
    }
    for (; i < n; i += stride) {
        const uint4 a = src[i];
        x ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    if (x == 0x9E3779B9u) sink[blockIdx.x & 1023] = x;
}

double mean_cycles(const uint64_t* h, int n) {
    double s = 0;
    for (int i = 0; i < n; ++i) s += static_cast<double>(h[i]);
    return s / n;
}

}  // namespace

// Results (per SIMD unless noted; cycles are shader clocks):
//   out[0]  cycles per v_mfma_i32_32x32x32_i8 (4 chains, 1 wave/SIMD)
//   out[1]  cycles per v_mfma_i32_16x16x64_i8 (8 chains)
//   out[2]  cycles per v_fma_f32 wave64 instruction (16 chains)
//   out[3]  cycles per cvt pair (v_cvt_f32_i32 + v_cvt_i32_f32 + add)
//   out[4+i] for i = 0..6: cycles per 32x32x32 MFMA with V = {0,2,4,6,7,8,12}
//           independent v_fma_f32 interleaved per MFMA in the same wave
//   out[11] MFMA cycles per instruction with a v_fma_f32 wave on the same SIMD
//   out[12] v_fma_f32 cycles per instruction with an MFMA wave on the same SIMD
//   out[13] LDS ds_read_b128 bytes per cycle per CU (4 waves)
//   out[14] shader clock in MHz (from the 100 MHz counter)
//   out[15] number of CUs
extern "C" int apex4_rho_probe(double* out, int n_out) {
    if (!out || n_out < 16) return -1;
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return -2;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -2;
    uint64_t* cyc_d = nullptr;
    int* sink = nullptr;
    const int nw = ncu * 8;
    if (hipMalloc(&cyc_d, sizeof(uint64_t) * nw) != hipSuccess) return -3;
    if (hipMalloc(&sink, sizeof(int) * 512) != hipSuccess) { (void)hipFree(cyc_d); return -3; }
    uint64_t* h = new uint64_t[nw];
    const size_t lds_hold = 96 * 1024;   // keeps a second workgroup off the CU
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(lds_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                        static_cast<int>(lds_hold));
    int rc = 0;
    auto run4 = [&](void (*k)(int, uint64_t*, int*), double per) -> double {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(lds_hold));
        hipLaunchKernelGGL(k, dim3(ncu), dim3(256), lds_hold, 0, 3, cyc_d, sink);
        if (hipDeviceSynchronize() != hipSuccess) { rc = -4; return 0; }
        (void)hipMemcpy(h, cyc_d, sizeof(uint64_t) * ncu * 4, hipMemcpyDeviceToHost);
        return mean_cycles(h, ncu * 4) / per;
    };
    out[0] = run4(mfma32_kernel<0>, ITERS * 4.0);
    out[1] = run4(mfma16_kernel, ITERS * 8.0);
    out[2] = run4(fma_kernel<256>, ITERS * 16.0);
    out[3] = run4(cvt_kernel, ITERS * 16.0);
    out[4] = run4(mfma32_kernel<0>, ITERS * 4.0);
    out[5] = run4(mfma32_kernel<2>, ITERS * 4.0);
    out[6] = run4(mfma32_kernel<4>, ITERS * 4.0);
    out[7] = run4(mfma32_kernel<6>, ITERS * 4.0);
    out[8] = run4(mfma32_kernel<7>, ITERS * 4.0);
    out[9] = run4(mfma32_kernel<8>, ITERS * 4.0);
    out[10] = run4(mfma32_kernel<12>, ITERS * 4.0);
    if (!rc) {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(split_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(lds_hold));
        hipLaunchKernelGGL(split_kernel, dim3(ncu), dim3(512), lds_hold, 0, 3, cyc_d, sink);
        if (hipDeviceSynchronize() != hipSuccess) rc = -4;
        (void)hipMemcpy(h, cyc_d, sizeof(uint64_t) * ncu * 8, hipMemcpyDeviceToHost);
        double mf = 0, va = 0;
        for (int b = 0; b < ncu; ++b)
            for (int w = 0; w < 8; ++w) (w < 4 ? mf : va) += static_cast<double>(h[b * 8 + w]);
        out[11] = mf / (ncu * 4.0) / (ITERS * 4.0);
        out[12] = va / (ncu * 4.0) / (ITERS * 2.0 * 16.0);
    }
    if (!rc) {
        const double cyc_per_iter = run4(lds_kernel, ITERS);
        out[13] = cyc_per_iter > 0 ? (256.0 * 8 * 16) / cyc_per_iter : 0;   // bytes per iteration per CU
    }
    if (!rc) {
        (void)hipMemset(cyc_d, 0, sizeof(uint64_t) * 4);
        hipLaunchKernelGGL(clock_kernel, dim3(1), dim3(64), 0, 0, cyc_d);
        if (hipDeviceSynchronize() != hipSuccess) rc = -4;
        (void)hipMemcpy(h, cyc_d, sizeof(uint64_t) * 4, hipMemcpyDeviceToHost);
        out[14] = h[2] ? 100.0 * static_cast<double>(h[1]) / static_cast<double>(h[2]) : 0;
    }
    out[15] = ncu;
    delete[] h;
    (void)hipFree(cyc_d);
    (void)hipFree(sink);
    return rc;
}

// Sustained issue rates with several waves per SIMD (cycles per SIMD):
//   out[0] cycles per v_fma_f32 with 2 waves per SIMD
//   out[1] cycles per v_fma_f32 with 4 waves per SIMD
//   out[2 + i], i = 0..6: cycles per v_mfma_i32_32x32x32_i8 with 2 waves per
//          SIMD, each wave interleaving V = {0, 2, 4, 6, 8, 11, 16} independent
//          v_fma_f32 per MFMA
extern "C" int apex4_rho_probe_issue(double* out, int n_out) {
    if (!out || n_out < 9) return -1;
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return -2;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -2;
    uint64_t* cyc_d = nullptr;
    int* sink = nullptr;
    const int nw = ncu * 16;
    if (hipMalloc(&cyc_d, sizeof(uint64_t) * nw) != hipSuccess) return -3;
    if (hipMalloc(&sink, sizeof(int) * 256) != hipSuccess) { (void)hipFree(cyc_d); return -3; }
    uint64_t* h = new uint64_t[nw];
    const size_t hold = 96 * 1024;
    int rc = 0;
    // Per-SIMD cycles per instruction: the waves of a workgroup start together
    // (barrier), so the slowest wave's count is the elapsed time of its SIMD;
    // divide by the instructions all waves of that SIMD issued.
    auto run = [&](void (*k)(int, uint64_t*, int*), int threads, double per_wave) -> double {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                  static_cast<int>(hold));
        hipLaunchKernelGGL(k, dim3(ncu), dim3(threads), hold, 0, 3, cyc_d, sink);
        if (hipDeviceSynchronize() != hipSuccess) { rc = -4; return 0; }
        const int waves = threads / 64;
        (void)hipMemcpy(h, cyc_d, sizeof(uint64_t) * ncu * waves, hipMemcpyDeviceToHost);
        double sum = 0;
        for (int b = 0; b < ncu; ++b) {
            uint64_t mx = 0;
            for (int w = 0; w < waves; ++w) mx = h[b * waves + w] > mx ? h[b * waves + w] : mx;
            sum += static_cast<double>(mx);
        }
        return sum / ncu / (per_wave * (waves / 4));
    };
    out[0] = run(fma_kernel<512>, 512, ITERS * 16.0);
    out[1] = run(fma_kernel<1024>, 1024, ITERS * 16.0);
    out[2] = run(mfma32_kernel<0, 512>, 512, ITERS * 4.0);
    out[3] = run(mfma32_kernel<2, 512>, 512, ITERS * 4.0);
    out[4] = run(mfma32_kernel<4, 512>, 512, ITERS * 4.0);
    out[5] = run(mfma32_kernel<6, 512>, 512, ITERS * 4.0);
    out[6] = run(mfma32_kernel<8, 512>, 512, ITERS * 4.0);
    out[7] = run(mfma32_kernel<11, 512>, 512, ITERS * 4.0);
    out[8] = run(mfma32_kernel<16, 512>, 512, ITERS * 4.0);
    delete[] h;
    (void)hipFree(cyc_d);
    (void)hipFree(sink);
    return rc;
}

// Copy nbytes (a multiple of 16, both pointers 16-byte aligned device memory)
// from src to dst on `stream`.
extern "C" int apex4_copy_probe(const void* src, void* dst, int64_t nbytes, void* stream) {
    if (!src || !dst || nbytes < 0 || (nbytes & 15)) return -1;
    const int64_t n = nbytes / 16;
    if (n == 0) return 0;
    hipLaunchKernelGGL(copy_kernel, dim3(4096), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const uint4*>(src), static_cast<uint4*>(dst), n);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

// Read nbytes (a multiple of 16; src 16-byte aligned device memory) on
// `stream`; sink: device memory of at least 4096 bytes (written only for one
// magic xor of the data, which the callers' data does not produce).
extern "C" int apex4_read_probe(const void* src, int64_t nbytes, void* sink, void* stream) {
    if (!src || !sink || nbytes < 0 || (nbytes & 15) || (reinterpret_cast<uintptr_t>(src) & 15)) return -1;
    const int64_t n = nbytes / 16;
    if (n == 0) return 0;
    hipLaunchKernelGGL(read_kernel, dim3(8192), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const uint4*>(src), n, static_cast<uint32_t*>(sink));
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

// Extended probes (cycles per SIMD unless noted):
//   out[0] cycles per MFMA, 1 dependent chain per wave, 1 wave per SIMD
//   out[1] cycles per MFMA, 2 chains per wave, 1 wave per SIMD
//   out[2] cycles per MFMA per wave, 1 chain per wave, 2 waves per SIMD
//   out[3] LDS ds_read_b128 bytes per cycle per CU, 4 waves x 16 in flight
//   out[4] same, 8 waves x 16 in flight
extern "C" int apex4_rho_probe_ext(double* out, int n_out) {
    if (!out || n_out < 5) return -1;
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return -2;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -2;
    uint64_t* cyc_d = nullptr;
    int* sink = nullptr;
    const int nw = ncu * 8;
    if (hipMalloc(&cyc_d, sizeof(uint64_t) * nw) != hipSuccess) return -3;
    if (hipMalloc(&sink, sizeof(int) * 512) != hipSuccess) { (void)hipFree(cyc_d); return -3; }
    uint64_t* h = new uint64_t[nw];
    const size_t hold = 96 * 1024;
    int rc = 0;
    auto run = [&](void (*k)(int, uint64_t*, int*), int threads, double per) -> double {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                  static_cast<int>(hold));
        hipLaunchKernelGGL(k, dim3(ncu), dim3(threads), hold, 0, 3, cyc_d, sink);
        if (hipDeviceSynchronize() != hipSuccess) { rc = -4; return 0; }
        (void)hipMemcpy(h, cyc_d, sizeof(uint64_t) * nw, hipMemcpyDeviceToHost);
        const int waves = threads / 64;
        double sum = 0;
        for (int b = 0; b < ncu; ++b)
            for (int w = 0; w < waves; ++w) sum += static_cast<double>(h[b * 8 + w]);
        return sum / (ncu * waves) / per;
    };
    out[0] = run(mfma_chain_kernel<1>, 256, ITERS * 1.0);
    out[1] = run(mfma_chain_kernel<2>, 256, ITERS * 2.0);
    out[2] = run(mfma_chain_kernel<1>, 512, ITERS * 1.0);
    const double c4 = run(lds16_kernel<4>, 256, ITERS / 2);
    out[3] = c4 > 0 ? (4 * 64 * 16 * 16.0) / c4 : 0;
    const double c8 = run(lds16_kernel<8>, 512, ITERS / 2);
    out[4] = c8 > 0 ? (8 * 64 * 16 * 16.0) / c8 : 0;
    delete[] h;
    (void)hipFree(cyc_d);
    (void)hipFree(sink);
    return rc;
}
