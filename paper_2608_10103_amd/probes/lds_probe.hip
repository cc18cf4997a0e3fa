// lds_probe.hip - LDS measurements behind the kernels' LDS layout (MI355X).
//
// lds_read_swizzle: every wave of a 512-thread workgroup repeatedly reads the
//   operand runs of four 32x32 MFMA blocks from LDS exactly as the GEMM
//   kernels do (lane l: row q0 + l % 32, 16-byte chunk c0 + l / 32 of rows of
//   `row_bytes`), with chunk c of row q stored at slot
//   c ^ (((q >> sa) ^ (q >> sb)) & (chunks - 1)) (sb < 0: (q >> sa) & ...).
//   Its run time ranks swizzles by LDS bank conflicts.
// lds_read_with_writes: eight 1 KiB operand reads per wave per iteration plus,
//   per iteration, one extra LDS write of the given kind: 0 none, 1 a 16-byte
//   per lane direct-to-LDS load (1 KiB), 2 a 4-byte per lane one (256 bytes),
//   3 a ds_write_b128 (1 KiB). Its run time shows what a write costs the reads.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

__global__ __launch_bounds__(512, 1) void lds_read_swizzle(int row_bytes, int sa, int sb, int iters,
                                                          int *sink) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[65536];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ch = row_bytes / 16;
    for (int i = threadIdx.x; i < 65536 / 16; i += 512)
        *reinterpret_cast<i32x4 *>(lds + i * 16) = i32x4{i, sa, sb, row_bytes};
    __syncthreads();
    int off[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int q = (wave & 1) * 128 + (j & 3) * 32 + (lane & 31);
        const int c = ((lane >> 5) + 2 * (j >> 2)) % ch;
        int s = q >> sa;
        if (sb >= 0) s ^= q >> sb;
        s &= ch - 1;
        off[j] = (q * row_bytes + ((c ^ s) << 4)) & 65535;
    }
    i32x4 acc = {0, 0, 0, 0};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc ^= *reinterpret_cast<const i32x4 *>(lds + off[j]);
        asm volatile("" : "+v"(acc)::"memory");
    }
    if (acc[0] == 0x12345678 && acc[1] == 7) sink[0] = acc[2];
}

template <int KIND>
__global__ __launch_bounds__(512, 1) void lds_read_with_writes(const uint8_t *__restrict__ src,
                                                              int iters, int *sink) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[131072];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int i = threadIdx.x; i < 65536 / 16; i += 512)
        *reinterpret_cast<i32x4 *>(lds + i * 16) = i32x4{i, 1, 2, 3};
    __syncthreads();
    const uint8_t *base = lds + wave * 8192 + lane * 16;
    i32x4 acc = {0, 0, 0, 0};
    for (int it = 0; it < iters; ++it) {
        uint8_t *dst = lds + 65536 + (wave * 4 + (it & 3)) * 1024;
        // 1 MiB source window, 1 KiB per wave-instruction, in bounds for any it
        const uint8_t *g = src + (((long)blockIdx.x * 64 + (it & 63)) * 1024 & ((1 << 20) - 1)) + lane * 16;
        if constexpr (KIND == 1) __builtin_amdgcn_global_load_lds(g, (lds_void *)dst, 16, 0, 0);
        if constexpr (KIND == 2) __builtin_amdgcn_global_load_lds(g, (lds_void *)dst, 4, 0, 0);
        if constexpr (KIND == 3) *reinterpret_cast<i32x4 *>(dst + lane * 16) = acc;
#pragma unroll
        for (int j = 0; j < 8; ++j) acc ^= *reinterpret_cast<const i32x4 *>(base + j * 1024);
        asm volatile("" : "+v"(acc)::"memory");
    }
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
    if (acc[0] == 0x12345678 && acc[1] == 7) sink[0] = acc[2];
}

extern "C" int probe_lds_read_swizzle(int row_bytes, int sa, int sb, int iters, int grid, int *sink,
                                      hipStream_t s) {
    if (row_bytes != 64 && row_bytes != 128) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(lds_read_swizzle, dim3(grid), dim3(512), 0, s, row_bytes, sa, sb, iters, sink);
    return (int)hipGetLastError();
}

extern "C" int probe_lds_read_with_writes(int kind, const void *src_1mib, int iters, int grid, int *sink,
                                          hipStream_t s) {
    const void *f[] = {(const void *)&lds_read_with_writes<0>, (const void *)&lds_read_with_writes<1>,
                       (const void *)&lds_read_with_writes<2>, (const void *)&lds_read_with_writes<3>};
    if (kind < 0 || kind > 3) return (int)hipErrorInvalidValue;
    const uint8_t *p = static_cast<const uint8_t *>(src_1mib);
    void *args[] = {&p, &iters, &sink};
    return (int)hipLaunchKernel(f[kind], dim3(grid), dim3(512), args, 0, s);
}
