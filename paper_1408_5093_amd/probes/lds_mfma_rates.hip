// lds_mfma_rates.hip -- per-CU LDS read bandwidth (conflict-free
// ds_read_b128, 4 waves per workgroup) and the issue rate of back-to-back
// independent v_mfma_f32_32x32x16_bf16 (8 accumulator chains per wave).
//
// Build and run (one MI355X):
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       paper_1408_5093_amd/probes/lds_mfma_rates.hip -o /tmp/lds_mfma_rates
//   /tmp/lds_mfma_rates
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

__global__ void __launch_bounds__(256) lds_read(int iters, uint32_t* out)
{
    __shared__ u32x4 L[8192];  // 128 KB
    const int t = threadIdx.x;
    for (int i = t; i < 8192; i += 256)
        L[i] = u32x4{(uint32_t)i, 1u, 2u, 3u};
    __syncthreads();
    u32x4 acc = {0, 0, 0, 0};
    int base = (t >> 6) * 2048 + (t & 63);
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int q = 0; q < 8; ++q)
            acc ^= L[(base + q * 64) & 8191];
        base += 8 * 64;
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x12345678u)
        out[0] = 1;
}

__global__ void __launch_bounds__(256) mfma_only(int iters, float* out)
{
    floatx16 c[8];
    for (int i = 0; i < 8; ++i)
        c[i] = floatx16{};
    bf16x8 a, b;
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(float)(threadIdx.x + i);
        b[i] = (__bf16)1.0f;
    }
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            c[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[i], 0, 0, 0);
    }
    float s = 0;
    for (int i = 0; i < 8; ++i)
        s += c[i][0];
    if (s == 123.f)
        out[0] = s;
}

int main()
{
    uint32_t* out;
    if (hipMalloc(&out, 64) != hipSuccess)
        return 1;
    hipEvent_t a, b;
    (void)hipEventCreate(&a);
    (void)hipEventCreate(&b);
    int cus = 0;
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0);
    const int iters = 4096;
    for (int grid : {256, 512}) {
        float ms = 0;
        for (int rep = 0; rep < 2; ++rep) {
            (void)hipEventRecord(a);
            hipLaunchKernelGGL(lds_read, dim3(grid), dim3(256), 0, 0, iters, out);
            (void)hipEventRecord(b);
            (void)hipEventSynchronize(b);
            (void)hipEventElapsedTime(&ms, a, b);
        }
        const double bytes = (double)grid * 256 * 16 * 8 * iters;
        printf("ds_read_b128, %4d workgroups: %6.1f B/ns per CU\n", grid,
               bytes / (ms * 1e6) / cus);
    }
    for (int grid : {256, 512, 1024}) {
        float ms = 0;
        for (int rep = 0; rep < 2; ++rep) {
            (void)hipEventRecord(a);
            hipLaunchKernelGGL(mfma_only, dim3(grid), dim3(256), 0, 0, iters, (float*)out);
            (void)hipEventRecord(b);
            (void)hipEventSynchronize(b);
            (void)hipEventElapsedTime(&ms, a, b);
        }
        const double n = (double)grid * 4 * 8 * iters;
        printf("32x32x16 bf16 MFMA, %4d workgroups: %7.1f TFLOP/s, %.1f ns per instruction per SIMD\n",
               grid, n * 32768.0 / (ms * 1e-3) / 1e12, (ms * 1e6) / (n / (cus * 4.0)));
    }
    return 0;
}
