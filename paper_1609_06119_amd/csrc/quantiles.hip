// Equal-frequency bin boundaries on the device (section 2.2): boundary k of
// feature j is the value of rank floor(k n / B) of the feature's n values.
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
__global__ __launch_bounds__(256) void quantile_keys_kernel(const float *__restrict__ x,
                                                            int64_t ldx, int64_t n, int j0, int dj,
                                                            uint64_t *__restrict__ keys,
                                                            int *__restrict__ err) {
    const int64_t total = (int64_t)dj * n;
    int nan = 0;
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t jj = t / n, i = t - jj * n;
        const uint32_t b = __float_as_uint(x[(int64_t)(j0 + jj) * ldx + i]);
        nan |= (b & 0x7fffffffu) > 0x7f800000u;
        keys[t] = ((uint64_t)jj << 32) | order_key(b);
    }
    if (nan) atomicOr(err, kErrNan);
}

// bounds[(j0 + jj) * (B - 1) + k - 1] = value of rank floor(k n / B) of
// feature j0 + jj, from the sorted keys
__global__ __launch_bounds__(256) void quantile_pick_kernel(const uint64_t *__restrict__ sorted,
                                                            int64_t n, int j0, int dj, int n_bins,
                                                            float *__restrict__ bounds) {
    const int nb = n_bins - 1;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < dj * nb; t += gridDim.x * blockDim.x) {
        const int jj = t / nb, k = t - jj * nb + 1;
        const int64_t r = ((int64_t)k * n) / n_bins;
        const uint32_t key = (uint32_t)sorted[(int64_t)jj * n + r];
        bounds[(size_t)(j0 + jj) * nb + (k - 1)] = __uint_as_float(order_key_inverse(key));
    }
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
                                      uint64_t *keys_b, void *temp, float *bounds, int *err,
                                      hipStream_t s) {
    for (int j0 = 0; j0 < d; j0 += qs.batch_features) {
        const int dj = std::min(qs.batch_features, d - j0);
        const int64_t total = (int64_t)dj * n;
        const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
        quantile_keys_kernel<<<blocks, 256, 0, s>>>(x, ldx, n, j0, dj, keys_a, err);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        rocprim::double_buffer<uint64_t> db(keys_a, keys_b);
        size_t temp_bytes = qs.temp_bytes;
        e = rocprim::radix_sort_keys(temp, temp_bytes, db, (size_t)total, 0u,
                                     32u + (unsigned)bits_for(dj), s);
        if (e != hipSuccess) return e;
        const int picks = dj * (n_bins - 1);
        quantile_pick_kernel<<<(picks + 255) / 256, 256, 0, s>>>(db.current(), n, j0, dj, n_bins,
                                                                 bounds);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace fbdt
