// Launch entry of the PAM matrix products (their kernel, for float32 and
// bfloat16 operands, is pam_gemm_dma_kernel in pam_gemm_dma.hip), the
// reductions that add the K slices of split-K plans in a fixed order, the
// fill of k == 0 products, and the static split-K scratch of the entry point
// that allocates nothing.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>

#include "pam_internal.h"

namespace pamk {

// ---------------------------------------------------------------------------
// PAM matrix products: the kernel is in pam_gemm_dma.hip
// ---------------------------------------------------------------------------

hipError_t launch_pam_gemm(int tile_m, int tile_n, int kgroups, bool trans_a, bool trans_b, bool bf16,
                           const GemmParams &p, hipStream_t stream) {
    const int64_t items = (int64_t)p.whole + (int64_t)p.split_tiles * p.splits;
    if (items <= 0 || items > kMaxLaunchItems)
        return hipErrorInvalidValue;
    return launch_pam_gemm_dma(tile_m, tile_n, kgroups, trans_a, trans_b, bf16, p, stream);
}

// ---------------------------------------------------------------------------
// Split-K reduction and k == 0 fill
// ---------------------------------------------------------------------------

// Four outputs to 16-byte aligned memory: the final C with the non-temporal
// hint (written once), split partial sums without it (the reduce reads them
// back soon, mostly from cache).
__device__ __forceinline__ void store_out4(float *p, float a, float b, float c, float d, bool final_c) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const f32x4 v = {a, b, c, d};
    if (final_c)
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(p));
    else
        *reinterpret_cast<f32x4 *>(p) = v;
}

__global__ void __launch_bounds__(256) splitk_reduce_kernel(const float *__restrict__ W, float *__restrict__ C,
                                                            int32_t m, int32_t n, int64_t ldc, int64_t strideC,
                                                            int32_t splits, int64_t total) {
    const int64_t mn = (int64_t)m * n;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        const int64_t b = idx / mn;
        const int64_t r = idx - b * mn;
        const int64_t i = r / n;
        const int64_t j = r - i * n;
        const float *w = W + b * splits * mn + r;
        float s = 0.0f;
        for (int q = 0; q < splits; ++q)
            s += w[q * mn];
        C[b * strideC + i * ldc + j] = s;
    }
}

// Each workgroup adds the K slices of a 256 x 4-output part of one split
// tile (grid-stride over the parts); each thread four consecutive outputs,
// slice by slice.
__global__ void __launch_bounds__(256) split_tile_reduce_kernel(GemmParams p, int bm, int bn) {
    const int gpr = bn / 4;                      // four-output groups per tile row
    const int parts = bm * bn / 4 / 256;         // parts per tile
    const int64_t tile_elems = (int64_t)bm * bn;
    const int64_t slice = (int64_t)p.split_tiles * tile_elems;
    const int64_t nparts = (int64_t)p.split_tiles * parts;
    for (int64_t b = blockIdx.x; b < nparts; b += gridDim.x) {
        const int64_t t = b / parts;
        const int g = (int)(b % parts) * 256 + threadIdx.x;
        const int64_t tile_lin = p.whole + t;
        const int64_t bz = tile_lin / p.tiles;
        const int tile = (int)(tile_lin % p.tiles);
        const int m0 = (tile / p.tiles_n) * bm;
        const int n0 = (tile % p.tiles_n) * bn;
        const int r = g / gpr;
        const int c = (g % gpr) * 4;
        if (m0 + r >= p.m || n0 + c >= p.n)
            continue;
        const float *w = p.W + t * tile_elems + r * bn + c;
        float4 sum = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        // Eight slices' loads in flight before their adds (in slice order):
        // a thread's loads are independent, only the sum is sequential.
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        int q = 0;
        for (; q + 8 <= p.splits; q += 8) {
            f32x4 x[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                x[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(w + (q + u) * slice));
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                sum.x += x[u].x;
                sum.y += x[u].y;
                sum.z += x[u].z;
                sum.w += x[u].w;
            }
        }
        for (; q < p.splits; ++q) {
            const f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(w + q * slice));
            sum.x += x.x;
            sum.y += x.y;
            sum.z += x.z;
            sum.w += x.w;
        }
        float *crow = p.C + bz * p.strideC + (int64_t)(m0 + r) * p.ldc + n0;
        if (p.vec_c && n0 + c + 3 < p.n) {
            store_out4(crow + c, sum.x, sum.y, sum.z, sum.w, true);
        } else {
            const float sv[4] = {sum.x, sum.y, sum.z, sum.w};
            for (int j = 0; j < 4; ++j)
                if (n0 + c + j < p.n)
                    crow[c + j] = sv[j];
        }
    }
}

hipError_t launch_split_tile_reduce(int tile_m, int tile_n, const GemmParams &p, hipStream_t stream) {
    if (p.split_tiles <= 0)
        return hipSuccess;
    const int64_t parts = (int64_t)p.split_tiles * (tile_m * tile_n / 4 / 256);
    const int64_t blocks = std::min<int64_t>(parts, 256 * 32);
    hipLaunchKernelGGL(split_tile_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, p, tile_m, tile_n);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float *W, float *C, int32_t m, int32_t n, int64_t ldc, int64_t strideC,
                                int32_t splits, int64_t batch, hipStream_t stream) {
    const int64_t total = batch * (int64_t)m * n;
    if (total <= 0)
        return hipSuccess;
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 256 * 32);
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, W, C, m, n, ldc, strideC,
                       splits, total);
    return hipGetLastError();
}

__global__ void __launch_bounds__(256) fill_zero_kernel(float *__restrict__ C, int32_t m, int32_t n, int64_t ldc,
                                                        int64_t strideC, int64_t total) {
    const int64_t mn = (int64_t)m * n;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        const int64_t b = idx / mn;
        const int64_t r = idx - b * mn;
        const int64_t i = r / n;
        const int64_t j = r - i * n;
        C[b * strideC + i * ldc + j] = 0.0f;
    }
}

hipError_t launch_fill_zero(float *C, int32_t m, int32_t n, int64_t ldc, int64_t strideC, int64_t batch,
                            hipStream_t stream) {
    const int64_t total = batch * (int64_t)m * n;
    if (total <= 0)
        return hipSuccess;
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 256 * 32);
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, C, m, n, ldc, strideC, total);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Static split-K scratch of pam_gemm_batched_noalloc
// ---------------------------------------------------------------------------

// File-scope device memory: every device the library runs on holds one copy
// until the process ends.  Host code must not pass `scratch` itself to a
// kernel or a copy (on the host it names a stand-in, not device memory): the
// device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 256;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t scratch_address(void **out) {
    *out = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        // Once per device, with that device current (hipGetDevice above).
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (ptr == nullptr)
            return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace pamk
