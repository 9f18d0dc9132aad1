// copy_patterns.hip -- throughput of 16-byte-per-lane loads from an
// L2-resident buffer by access pattern, as LDS DMA (buffer_load ... lds) and
// as loads into registers.  One wave instruction reads 1 KB: `rows` rows of
// 1024 / rows bytes at a row stride, lanes either row-fastest (lane l -> row
// l % rows) or chunk-fastest (lane l -> row l / (64 / rows)), the latter
// optionally with the chunks of a row XOR-permuted.
//
// Build and run (one MI355X):
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       paper_1408_5093_amd/probes/copy_patterns.hip -o /tmp/copy_patterns
//   /tmp/copy_patterns
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* b, uint32_t n)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(b), (short)0, (int)n, 0x00020000);
}

// byte offset of lane l: mode 0 row-fastest, 1 chunk-fastest, 2 chunk-fastest
// with the chunks of each row XOR-permuted
__device__ __forceinline__ uint32_t lane_off(int l, int rows, int stride, int mode)
{
    const int cpr = 64 / rows;
    if (mode == 0)
        return (uint32_t)((l % rows) * stride + (l / rows) * 16);
    const int row = l / cpr, ch = l % cpr;
    const int swz = mode == 2 ? (row & (cpr - 1)) : 0;
    return (uint32_t)(row * stride + (ch ^ swz) * 16);
}

template <bool DMA>
__global__ void __launch_bounds__(256)
probe(const uint32_t* X, uint32_t nbytes, int rows, int stride, int mode, int iters,
      uint32_t* out)
{
    __shared__ u32x4 L[4][8][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const __amdgpu_buffer_rsrc_t r = rsrc(X, nbytes);
    const uint32_t lo = lane_off(lane, rows, stride, mode);
    const uint32_t span = (uint32_t)(rows * stride);
    uint32_t base = (uint32_t)((blockIdx.x * 4 + w) * 8) * span % (nbytes - 8 * span);
    u32x4 acc = {0, 0, 0, 0};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const uint32_t off = base + q * span + lo;
            if (DMA)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)&L[w][q][0], 16, off, 0, 0,
                                                         0);
            else
                acc ^= __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
        }
        if (DMA)
            __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        base += 8 * span;
        if (base + 8 * span > nbytes)
            base = (base + 4096) % (nbytes / 2);
    }
    if (DMA)
        acc = L[w][lane & 7][lane];
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x12345678u)
        out[0] = 1;
}

int main()
{
    const uint32_t nb = 2u << 20;  // 2 MB: L2-resident
    uint32_t *X, *out;
    if (hipMalloc(&X, nb) != hipSuccess || hipMalloc(&out, 4) != hipSuccess)
        return 1;
    (void)hipMemset(X, 1, nb);
    hipEvent_t a, b;
    (void)hipEventCreate(&a);
    (void)hipEventCreate(&b);
    int cus = 0, clk = 0;
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0);
    (void)hipDeviceGetAttribute(&clk, hipDeviceAttributeClockRate, 0);
    const int grid = 4096, iters = 64;
    struct P { int rows, stride, mode; } pats[] = {
        {64, 16, 0},   {16, 512, 0},  {64, 512, 0},  {8, 512, 1},   {8, 512, 2},
        {8, 4608, 2},  {16, 512, 1},  {16, 4608, 2}, {32, 512, 1}};
    printf("kind  rows x bytes  stride  lanes          B/clk/CU  (clock %d MHz, %d CUs)\n",
           clk / 1000, cus);
    for (int dma = 1; dma >= 0; --dma)
        for (const P& p : pats) {
            float ms = 0;
            for (int rep = 0; rep < 2; ++rep) {
                (void)hipEventRecord(a);
                if (dma)
                    hipLaunchKernelGGL(probe<true>, dim3(grid), dim3(256), 0, 0, X, nb, p.rows,
                                       p.stride, p.mode, iters, out);
                else
                    hipLaunchKernelGGL(probe<false>, dim3(grid), dim3(256), 0, 0, X, nb, p.rows,
                                       p.stride, p.mode, iters, out);
                (void)hipEventRecord(b);
                (void)hipEventSynchronize(b);
                (void)hipEventElapsedTime(&ms, a, b);
            }
            const double bytes = (double)grid * 4 * iters * 8 * 1024;
            const char* lanes = p.mode == 0 ? "row-fastest" : p.mode == 1 ? "chunk-fastest"
                                                                         : "chunk-fastest xor";
            printf("%s  %2d x %4d     %5d   %-17s %6.1f\n", dma ? "dma " : "vgpr", p.rows,
                   1024 / p.rows, p.stride, lanes,
                   bytes / (ms * 1e-3) / cus / ((double)clk * 1e3));
        }
    return 0;
}
