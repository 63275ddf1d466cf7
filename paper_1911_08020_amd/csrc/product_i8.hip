// INT8 retained weights (section 4.2's storage accounting assumes weights quantised
// to INT8): per-row symmetric codes and scales, and the DARB products on them
// (kernels and launch templates in product_common.h).
//
// Quantisation of row r, over its retained values v (fp32, or fp16 widened
// exactly): a = max |v|, inv = 127 / a, q = rint(v * inv) clamped to [-127, 127],
// scale s_r = a / 127; each step is one correctly rounded fp32 operation, so the
// codes do not depend on the order of any reduction (the max is exact).  Rows with
// a < 2^-120, where 127 / a would overflow, get s_r = 0 and q = 0.
#include "product_common.h"

namespace darb {
namespace {

constexpr int kQuantThreads = 256;
constexpr int kQuantUnroll = 8;
constexpr float kI8MinAbsmax = 0x1p-120f;

template <typename Tw>
__device__ __forceinline__ float value_f32(const Tw *v, int64_t i) { return to_f32<Tw>(v[i]); }

// One wave per storage-order row: the row's largest magnitude (xor-butterfly max,
// exact in any order), then its codes; the scale goes to the row's original index.
template <typename Tw>
__global__ __launch_bounds__(kQuantThreads) void quantize_i8_kernel(
    const Tw *__restrict__ values, int8_t *__restrict__ codes, float *__restrict__ scales,
    const int32_t *__restrict__ perm, int64_t M, BinTable bins) {
    const int64_t i = int64_t(blockIdx.x) * (kQuantThreads / kWave) + threadIdx.x / kWave;
    if (i >= M) return;                                   // wave-uniform, no barrier below
    const int lane = int(threadIdx.x) & (kWave - 1);
    int g = 0;
#pragma unroll
    for (int b = 1; b < kMaxBins; ++b)
        if (b < bins.nbins && i >= bins.first_row[b]) g = b;
    const int64_t nblk = pick(bins.nblk, g);
    const int64_t e0 = pick(bins.first_elem, g) + (i - pick(bins.first_row, g)) * nblk;

    // kQuantUnroll loads in flight per lane (indices clamped into the row, masked)
    float a = 0.0f;
    for (int64_t k0 = lane; k0 < nblk; k0 += kQuantUnroll * kWave) {
        float v[kQuantUnroll];
#pragma unroll
        for (int u = 0; u < kQuantUnroll; ++u) {
            const int64_t k = k0 + u * kWave;
            v[u] = value_f32(values, e0 + (k < nblk ? k : nblk - 1));
        }
#pragma unroll
        for (int u = 0; u < kQuantUnroll; ++u) a = fmaxf(a, fabsf(v[u]));
    }
    for (int m = kWave / 2; m >= 1; m >>= 1) a = fmaxf(a, __shfl_xor(a, m, kWave));

    const bool live = a >= kI8MinAbsmax;
    const float inv = live ? __fdiv_rn(127.0f, a) : 0.0f;
    for (int64_t k0 = lane; k0 < nblk; k0 += kQuantUnroll * kWave) {
        float v[kQuantUnroll];
#pragma unroll
        for (int u = 0; u < kQuantUnroll; ++u) {
            const int64_t k = k0 + u * kWave;
            v[u] = value_f32(values, e0 + (k < nblk ? k : nblk - 1));
        }
#pragma unroll
        for (int u = 0; u < kQuantUnroll; ++u) {
            const int64_t k = k0 + u * kWave;
            const float q = rintf(__fmul_rn(v[u], inv));
            if (k < nblk) codes[e0 + k] = int8_t(fminf(fmaxf(q, -127.0f), 127.0f));
        }
    }
    if (lane == 0) scales[perm[i]] = live ? __fdiv_rn(a, 127.0f) : 0.0f;
}

template <typename Tw>
hipError_t launch_quantize_t(const darb_plan &p, const void *values, int8_t *codes,
                             float *scales, hipStream_t s) {
    constexpr int rows_per_block = kQuantThreads / kWave;
    const int64_t blocks = (p.M + rows_per_block - 1) / rows_per_block;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((quantize_i8_kernel<Tw>), dim3(unsigned(blocks)), dim3(kQuantThreads), 0,
                       s, static_cast<const Tw *>(values), codes, scales, p.d_perm, p.M, p.bins);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize_i8(const darb_plan &p, int wdtype, const void *values, int8_t *codes,
                              float *scales, hipStream_t s) {
    if (wdtype == DARB_F32) return launch_quantize_t<float>(p, values, codes, scales, s);
    return launch_quantize_t<__half>(p, values, codes, scales, s);
}

hipError_t launch_spmv_i8(const darb_plan &p, const int8_t *codes, const float *scales,
                          const uint8_t *offsets, const uint32_t *packed, int xdtype,
                          const void *x, float *y, hipStream_t s) {
    if (xdtype == DARB_F16)
        return launch_spmv_form<int8_t, __half>(p, codes, offsets, packed, x, y, scales, s);
    return launch_spmv_form<int8_t, float>(p, codes, offsets, packed, x, y, scales, s);
}

hipError_t launch_spmm_i8(const darb_plan &p, const int8_t *codes, const float *scales,
                          const uint8_t *offsets, const uint32_t *packed, int xdtype, int64_t B,
                          const void *X, int64_t ldx, float *Y, int64_t ldy, hipStream_t s) {
    if (xdtype == DARB_F16)
        return launch_spmm_form<int8_t, __half>(p, codes, offsets, packed, B, X, ldx, Y, ldy,
                                                scales, s);
    return launch_spmm_form<int8_t, float>(p, codes, offsets, packed, B, X, ldx, Y, ldy, scales,
                                           s);
}

}  // namespace darb
