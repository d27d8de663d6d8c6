// Equal-frequency bin boundaries on the device (section 2.2): boundary k of
// feature j is the value of rank floor(k m / B) among the feature's m
// non-NaN values (NaN values are missing, section 4.2).
// Each value becomes a 64-bit key, the feature index (within a batch of
// features) above an order-preserving 32-bit image of the float, so that one
// device-wide radix sort (rocPRIM) orders every feature of the batch at once;
// the boundaries are then read off at their ranks.
#include "fbdt_internal.h"

#include <hip/hip_runtime.h>

#include <rocprim/device/device_radix_sort.hpp>

namespace fbdt {
namespace {

// Order-preserving image of a non-NaN float: unsigned order of the image =
// numeric order of the floats (-0 sorts just below +0).
__device__ __forceinline__ uint32_t order_key(uint32_t b) {
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ uint32_t order_key_inverse(uint32_t k) {
    return (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
}

// keys[jj * n + i] = jj << 32 | order_key(x[j0 + jj][i]) for jj < dj
// (blockIdx.y = jj); nan_count[jj] += the feature's NaN values, which sort
// after +inf
__global__ __launch_bounds__(256) void quantile_keys_kernel(
    const float *__restrict__ x, int64_t ldx, int64_t n, int j0, uint64_t *__restrict__ keys,
    unsigned long long *__restrict__ nan_count) {
    const int jj = blockIdx.y;
    unsigned long long nan = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t b = __float_as_uint(x[(int64_t)(j0 + jj) * ldx + i]);
        const bool is_nan = (b & 0x7fffffffu) > 0x7f800000u;
        nan += is_nan ? 1ull : 0ull;
        // every NaN, whatever its sign, sorts last
        keys[(int64_t)jj * n + i] = ((uint64_t)jj << 32) | (is_nan ? 0xffffffffu : order_key(b));
    }
    for (int off = warpSize / 2; off > 0; off >>= 1) nan += __shfl_down(nan, off);
    if (threadIdx.x % warpSize == 0 && nan) atomicAdd(&nan_count[jj], nan);
}

// bounds[(j0 + jj) * (B - 1) + k - 1] = value of rank floor(k m / B) among
// the m non-NaN values of feature j0 + jj (NaN sorts last), from the sorted
// keys; +inf when every value is NaN
__global__ __launch_bounds__(256) void quantile_pick_kernel(
    const uint64_t *__restrict__ sorted, int64_t n, int j0, int dj, int n_bins,
    const unsigned long long *__restrict__ nan_count, float *__restrict__ bounds) {
    const int nb = n_bins - 1;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < dj * nb; t += gridDim.x * blockDim.x) {
        const int jj = t / nb, k = t - jj * nb + 1;
        const int64_t m = n - (int64_t)nan_count[jj];
        float b = __uint_as_float(0x7f800000u);   // +inf
        if (m > 0) {
            const int64_t r = ((int64_t)k * m) / n_bins;
            b = __uint_as_float(order_key_inverse((uint32_t)sorted[(int64_t)jj * n + r]));
        }
        bounds[(size_t)(j0 + jj) * nb + (k - 1)] = b;
    }
}

__global__ void nan_flag_kernel(const unsigned long long *__restrict__ nan_count, int d,
                                int *__restrict__ err) {
    for (int j = threadIdx.x; j < d; j += blockDim.x)
        if (nan_count[j]) atomicOr(err, kErrNan);
}

int bits_for(int v) {   // bits needed to hold 0 .. v - 1
    int b = 0;
    while ((1 << b) < v) ++b;
    return b;
}

}  // namespace

int quantile_batch_features(int64_t n, int d) {
    int64_t dj = kQuantileBatchKeys / (n > 0 ? n : 1);
    if (dj < 1) dj = 1;
    if (dj > d) dj = d;
    return (int)dj;
}

hipError_t quantile_scratch(int64_t n, int d, QuantileScratch *qs) {
    const int dj = quantile_batch_features(n, d);
    const size_t keys = (size_t)dj * (size_t)n;
    rocprim::double_buffer<uint64_t> db(nullptr, nullptr);
    size_t temp = 0;
    const hipError_t e = rocprim::radix_sort_keys(nullptr, temp, db, keys, 0u,
                                                  32u + (unsigned)bits_for(dj));
    if (e != hipSuccess) return e;
    qs->batch_features = dj;
    qs->key_elems = keys;
    qs->temp_bytes = temp;
    return hipSuccess;
}

hipError_t launch_quantile_boundaries(const float *x, int64_t ldx, int64_t n, int d, int n_bins,
                                      const QuantileScratch &qs, uint64_t *keys_a,
                                      uint64_t *keys_b, void *temp,
                                      unsigned long long *nan_count, float *bounds, int *err,
                                      hipStream_t s) {
    hipError_t e = launch_fill_u32(nan_count, 0u, 2 * (size_t)d, s);
    if (e != hipSuccess) return e;
    for (int j0 = 0; j0 < d; j0 += qs.batch_features) {
        const int dj = std::min(qs.batch_features, d - j0);
        const int64_t total = (int64_t)dj * n;
        const dim3 grid((unsigned)std::min<int64_t>((n + 255) / 256, 2048), (unsigned)dj);
        quantile_keys_kernel<<<grid, 256, 0, s>>>(x, ldx, n, j0, keys_a, nan_count + j0);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        rocprim::double_buffer<uint64_t> db(keys_a, keys_b);
        size_t temp_bytes = qs.temp_bytes;
        e = rocprim::radix_sort_keys(temp, temp_bytes, db, (size_t)total, 0u,
                                     32u + (unsigned)bits_for(dj), s);
        if (e != hipSuccess) return e;
        const int picks = dj * (n_bins - 1);
        quantile_pick_kernel<<<(picks + 255) / 256, 256, 0, s>>>(db.current(), n, j0, dj, n_bins,
                                                                 nan_count + j0, bounds);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // NaN is an error with 256 bins (no room for the missing code)
    if (n_bins > kMissingCode) {
        nan_flag_kernel<<<1, 256, 0, s>>>(nan_count, d, err);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace fbdt
