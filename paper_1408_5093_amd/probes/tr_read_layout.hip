// tr_read_layout.hip -- lane layout of ds_read_b64_tr_b16: LDS holds
// element i = i (16-bit); lane l points at elements 4l .. 4l + 3 and prints
// the four values it receives.  In each group of 16 lanes, lane j receives
// element j % 4 of the rows of lanes 4i + j / 4, i = 0..3 (a 4 x 4 transpose
// of 4-element blocks), which the weight-gradient kernel uses to gather 4
// consecutive pixel rows of one channel.
//
// Build and run (one MI355X):
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       paper_1408_5093_amd/probes/tr_read_layout.hip -o /tmp/tr_read_layout
//   /tmp/tr_read_layout
#include <hip/hip_runtime.h>
#include <stdio.h>

typedef short short4v __attribute__((ext_vector_type(4)));

__global__ void probe(short* o)
{
    __shared__ short L[256];
    for (int i = threadIdx.x; i < 256; i += 64)
        L[i] = (short)i;
    __syncthreads();
    const int l = threadIdx.x;
    const short4v r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) short4v*)&L[4 * l]);
    for (int i = 0; i < 4; ++i)
        o[l * 4 + i] = r[i];
}

int main()
{
    short* o;
    if (hipMalloc(&o, 512) != hipSuccess)
        return 1;
    hipLaunchKernelGGL(probe, dim3(1), dim3(64), 0, 0, o);
    short h[256];
    (void)hipMemcpy(h, o, sizeof(h), hipMemcpyDeviceToHost);
    int bad = 0;
    for (int l = 0; l < 64; ++l)
        for (int i = 0; i < 4; ++i) {
            const int j = l % 16, src = 16 * (l / 16) + 4 * i + j / 4;
            bad += h[4 * l + i] != 4 * src + j % 4;
        }
    for (int l = 0; l < 16; ++l)
        printf("lane %2d: %4d %4d %4d %4d\n", l, h[4 * l], h[4 * l + 1], h[4 * l + 2], h[4 * l + 3]);
    printf("layout %s for all 64 lanes\n", bad ? "DIFFERS from the stated transpose" : "matches");
    return bad != 0;
}
