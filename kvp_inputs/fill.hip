// Device side of the seeded input generator (kvp_inputs): the same SplitMix64
// stream and Irwin-Hall(4) construction as the host module, so a device-filled
// tensor equals the host-generated one bit for bit.  Input generation only; it
// holds none of the attention or planner arithmetic.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z ^= z >> 30;
    z *= 0xBF58476D1CE4E5B9ull;
    z ^= z >> 27;
    z *= 0x94D049BB133111EBull;
    z ^= z >> 31;
    return z;
}

__device__ __forceinline__ float normal_at(uint64_t key, uint64_t idx, float scale) {
    const uint64_t h = mix64(key + (idx + 1ull) * 0x9E3779B97F4A7C15ull);
    const int s = (int)(h & 0xFFFF) + (int)((h >> 16) & 0xFFFF) + (int)((h >> 32) & 0xFFFF) +
                  (int)((h >> 48) & 0xFFFF);
    return __fmul_rn((float)(s - 131070), scale);
}

// dst element at (i0, i1, i2, i3) with dst strides ds[] gets the value of logical
// index sum(i_k * ls[k]).  dims: n[4].  Element type: 0 = bf16 (RNE), 1 = fp32.
__global__ void fill_kernel(void* dst, int kind, uint64_t key, float scale, int64_t n0, int64_t n1,
                            int64_t n2, int64_t n3, int64_t d0, int64_t d1, int64_t d2, int64_t d3,
                            uint64_t l0, uint64_t l1, uint64_t l2, uint64_t l3, int64_t total) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        int64_t r = t;
        const int64_t i3 = r % n3;
        r /= n3;
        const int64_t i2 = r % n2;
        r /= n2;
        const int64_t i1 = r % n1;
        const int64_t i0 = r / n1;
        const uint64_t idx = (uint64_t)i0 * l0 + (uint64_t)i1 * l1 + (uint64_t)i2 * l2 + (uint64_t)i3 * l3;
        const int64_t off = i0 * d0 + i1 * d1 + i2 * d2 + i3 * d3;
        const float v = normal_at(key, idx, scale);
        if (kind == 0)
            ((__bf16*)dst)[off] = (__bf16)v;
        else
            ((float*)dst)[off] = v;
    }
}

// Paged cache: element (b, h, pos, c) of the logical cache [B][g][POS][d] (logical index
// b * lb + h * lh + pos * d + c) for pos < npos[b], stored at page pt[b * stride + pos / 64],
// row pos % 64 of a head-major pool [g][n][64][d] (transposed = 0) or [g][n][d][64]
// (transposed = 1).
// Unmapped (negative) entries are skipped.
__global__ void fill_pages_kernel(void* dst, int kind, uint64_t key, float scale, const int32_t* pt,
                                  int stride, int n_pages, const int32_t* npos, int g, int d,
                                  int transposed, uint64_t lb, uint64_t lh, int64_t total) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        int64_t r = t;
        int c, row;
        if (transposed) {
            row = (int)(r % 64);
            r /= 64;
            c = (int)(r % d);
            r /= d;
        } else {
            c = (int)(r % d);
            r /= d;
            row = (int)(r % 64);
            r /= 64;
        }
        const int h = (int)(r % g);
        r /= g;
        const int j = (int)(r % stride);
        const int b = (int)(r / stride);
        const int pos = 64 * j + row;
        if (pos >= npos[b]) continue;
        const int pg = pt[(int64_t)b * stride + j];
        if (pg < 0 || pg >= n_pages) continue;
        const int64_t off = transposed ? (((int64_t)h * n_pages + pg) * d + c) * 64 + row
                                       : (((int64_t)h * n_pages + pg) * 64 + row) * d + c;
        const uint64_t idx = (uint64_t)b * lb + (uint64_t)h * lh + (uint64_t)pos * d + (uint64_t)c;
        const float v = normal_at(key, idx, scale);
        if (kind == 0)
            ((__bf16*)dst)[off] = (__bf16)v;
        else
            ((float*)dst)[off] = v;
    }
}

}  // namespace

extern "C" int kvpin_fill_pages(void* dst, int kind, uint64_t key, float scale, const int32_t* pt, int stride,
                                int n_pages, const int32_t* npos, int B, int g, int d, int transposed,
                                uint64_t lb, uint64_t lh, void* stream) {
    if (!dst || !pt || !npos || B < 1 || g < 1 || d < 1 || stride < 1 || n_pages < 1 || (kind != 0 && kind != 1))
        return -1;
    const int64_t total = (int64_t)B * stride * g * 64 * d;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(fill_pages_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, dst, kind,
                       key, scale, pt, stride, n_pages, npos, g, d, transposed, lb, lh, total);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

extern "C" int kvpin_fill(void* dst, int kind, uint64_t key, float scale, const int64_t* n,
                          const int64_t* dstride, const uint64_t* lstride, void* stream) {
    if (!dst || !n || !dstride || !lstride || (kind != 0 && kind != 1)) return -1;
    const int64_t total = n[0] * n[1] * n[2] * n[3];
    if (total <= 0) return 0;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, dst, kind,
                       key, scale, n[0], n[1], n[2], n[3], dstride[0], dstride[1], dstride[2],
                       dstride[3], lstride[0], lstride[1], lstride[2], lstride[3], total);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}
