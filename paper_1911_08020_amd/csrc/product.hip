// DARB products on gfx950: y = W_darb x (SpMV) and Y = W_darb X (SpMM).
//
// Only retained weights are read (section 2), and each retained weight's
// in-block offset selects the one activation it multiplies (section 3.2):
//     y[r] = sum_k v[r,k] * x[k * b_r + off[r,k]].
// The grouped layout makes every block-size group a dense [rows x nblk] array,
// so a group is streamed with plain coalesced vector loads.
//
// SpMV: a wave owns `lanes_per_row` lanes per row and 64 / lanes_per_row rows of
// one group; lanes stride over the row's vectors (16-byte value loads plus the
// matching offset bytes).  The loads of the first chunk are issued before the
// workgroup stages x into LDS, so HBM latency overlaps the staging; the gathers
// then hit LDS.  Per-row sums are combined by an xor butterfly over the row's
// lanes (fixed order, deterministic) and written to y in original row order.
//
// SpMM: lanes map to batch columns (X is [N x B] row-major, so one weight's
// activations X[c, :] are contiguous); a row's (value, column) pairs are loaded
// one per lane and broadcast across the row's lanes with shuffles.
#include <hip/hip_fp16.h>

#include "darb_internal.h"

namespace darb {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kVmax = 8;                         // vectors in flight per lane (SpMV)
constexpr int64_t kLdsMaxFloats = 16384;         // x staged in LDS up to 64 KiB

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<__half>(__half v) { return __half2float(v); }

template <typename Tw> struct WVec;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <> struct WVec<float> {
    static constexpr int VEC = 4;
    using V = f32x4;        // 4 values, 16 bytes
    using O = uint32_t;     // their 4 offset bytes
    __device__ static float get(const V &v, int i) { return v[i]; }
};
template <> struct WVec<__half> {
    static constexpr int VEC = 8;
    using V = u32x4;        // 8 fp16 values, 16 bytes
    using O = u32x2;        // their 8 offset bytes
    __device__ static float get(const V &v, int i) {
        const uint32_t w = v[i >> 1];
        const uint16_t h = (i & 1) ? uint16_t(w >> 16) : uint16_t(w & 0xFFFFu);
        return __half2float(__ushort_as_half(h));
    }
};

__device__ __forceinline__ uint32_t off_byte(uint32_t o, int i) { return (o >> (8 * i)) & 0xFFu; }
__device__ __forceinline__ uint32_t off_byte(u32x2 o, int i) {
    return (o[i >> 2] >> (8 * (i & 3))) & 0xFFu;
}

__device__ __forceinline__ int find_group(const ProductSchedule &s, int64_t wtile) {
    int g = 0;
    while (g + 1 < s.nbins && wtile >= s.tile_begin[g + 1]) ++g;
    return g;
}

template <typename Tw, typename Tx, bool LDS>
__global__ __launch_bounds__(kThreads) void spmv_kernel(
    const Tw *__restrict__ values, const uint8_t *__restrict__ offsets,
    const Tx *__restrict__ x, float *__restrict__ y, const int32_t *__restrict__ perm,
    int64_t N, BinTable bins, ProductSchedule sch) {
    using WV = WVec<Tw>;
    constexpr int VEC = WV::VEC;
    extern __shared__ float xs[];

    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wtile = int64_t(blockIdx.x) * kWaves + threadIdx.x / kWave;
    const bool active = wtile < sch.tile_begin[sch.nbins];
    const int g = find_group(sch, active ? wtile : 0);
    const int L = sch.lanes_per_row[g];
    const int lb = bins.log2b[g];
    const int64_t nblk = bins.nblk[g];
    const int64_t row_in_group = (wtile - sch.tile_begin[g]) * (kWave / L) + lane / L;
    const bool row_ok = active && row_in_group < bins.rows[g];
    const int sub = lane & (L - 1);
    const int64_t e0 = bins.first_elem[g] + row_in_group * nblk;
    const bool vec_path = sch.vec[g] == VEC;
    const int64_t nvec = vec_path ? nblk / VEC : nblk;
    const int64_t stride = int64_t(L) * kVmax;

    // first chunk of this lane's vectors, issued before x is staged
    typename WV::V wv[kVmax];
    typename WV::O ov[kVmax];
    if (vec_path) {
#pragma unroll
        for (int t = 0; t < kVmax; ++t) {
            const int64_t vi = sub + int64_t(t) * L;
            if (row_ok && vi < nvec) {
                wv[t] = __builtin_nontemporal_load(
                    reinterpret_cast<const typename WV::V *>(values + e0) + vi);
                ov[t] = *(reinterpret_cast<const typename WV::O *>(offsets + e0) + vi);
            }
        }
    }

    if (LDS) {
        for (int64_t c = threadIdx.x; c < N; c += kThreads) xs[c] = to_f32<Tx>(x[c]);
        __syncthreads();
    }
    // offsets produced by the encode always give c < N; the global path clamps
    // anyway so a malformed offset cannot read outside x
    auto xat = [&](int64_t c) -> float {
        return LDS ? xs[c] : to_f32<Tx>(x[c < N ? c : N - 1]);
    };

    float acc = 0.0f;
    if (vec_path) {
        for (int64_t base = 0;; base += stride) {
#pragma unroll
            for (int t = 0; t < kVmax; ++t) {
                const int64_t vi = base + sub + int64_t(t) * L;
                if (row_ok && vi < nvec) {
#pragma unroll
                    for (int q = 0; q < VEC; ++q) {
                        const int64_t k = vi * VEC + q;
                        const int64_t c = (k << lb) + off_byte(ov[t], q);
                        acc = fmaf(WV::get(wv[t], q), xat(c), acc);
                    }
                }
            }
            if (base + stride >= nvec) break;
#pragma unroll
            for (int t = 0; t < kVmax; ++t) {
                const int64_t vi = base + stride + sub + int64_t(t) * L;
                if (row_ok && vi < nvec) {
                    wv[t] = __builtin_nontemporal_load(
                        reinterpret_cast<const typename WV::V *>(values + e0) + vi);
                    ov[t] = *(reinterpret_cast<const typename WV::O *>(offsets + e0) + vi);
                }
            }
        }
    } else if (row_ok) {
        for (int64_t k = sub; k < nblk; k += L) {
            const int64_t c = (k << lb) + offsets[e0 + k];
            acc = fmaf(to_f32<Tw>(values[e0 + k]), xat(c), acc);
        }
    }

    for (int m = L >> 1; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, kWave);
    if (row_ok && sub == 0) y[perm[bins.first_row[g] + row_in_group]] = acc;
}

template <typename Tw, typename Tx>
__global__ __launch_bounds__(kThreads) void spmm_kernel(
    const Tw *__restrict__ values, const uint8_t *__restrict__ offsets,
    const Tx *__restrict__ X, int64_t ldx, int64_t B, float *__restrict__ Y, int64_t ldy,
    const int32_t *__restrict__ perm, int64_t N, BinTable bins, ProductSchedule sch) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wtile = int64_t(blockIdx.x) * kWaves + threadIdx.x / kWave;
    if (wtile >= sch.tile_begin[sch.nbins]) return;   // wave-uniform
    const int g = find_group(sch, wtile);
    const int L = sch.lanes_per_row[g];
    const int lb = bins.log2b[g];
    const int64_t nblk = bins.nblk[g];
    const int64_t t_in_group = wtile - sch.tile_begin[g];
    const int64_t row_tile = t_in_group / sch.col_slabs;
    const int64_t slab = t_in_group - row_tile * sch.col_slabs;
    const int64_t row_in_group = row_tile * (kWave / L) + lane / L;
    const bool row_ok = row_in_group < bins.rows[g];
    const int sub = lane & (L - 1);
    const int64_t col = slab * L + sub;
    const bool col_ok = col < B;
    const int64_t e0 = bins.first_elem[g] + row_in_group * nblk;

    float acc = 0.0f;
    for (int64_t kb = 0; kb < nblk; kb += L) {
        const int64_t k = kb + sub;
        float v_l = 0.0f;
        int c_l = 0;
        if (row_ok && k < nblk) {
            v_l = to_f32<Tw>(values[e0 + k]);
            c_l = int((k << lb) + offsets[e0 + k]);
        }
        const int cnt = int(nblk - kb < L ? nblk - kb : L);
        for (int t = 0; t < cnt; ++t) {
            const float v = __shfl(v_l, t, L);
            int c = __shfl(c_l, t, L);
            c = c < N ? c : N - 1;                 // see the note in spmv_kernel
            if (row_ok && col_ok) acc = fmaf(v, to_f32<Tx>(X[int64_t(c) * ldx + col]), acc);
        }
    }
    if (row_ok && col_ok) Y[int64_t(perm[bins.first_row[g] + row_in_group]) * ldy + col] = acc;
}

template <typename Tw>
ProductSchedule spmv_schedule(const darb_plan &p, const void *values, const uint8_t *offsets) {
    constexpr int VEC = WVec<Tw>::VEC;
    ProductSchedule s{};
    s.nbins = p.bins.nbins;
    s.col_slabs = 1;
    int64_t tiles = 0;
    const bool ptr_ok = (reinterpret_cast<uintptr_t>(values) % 16 == 0) &&
                        (reinterpret_cast<uintptr_t>(offsets) % VEC == 0);
    for (int g = 0; g < s.nbins; ++g) {
        const int64_t nblk = p.bins.nblk[g];
        const bool vec = ptr_ok && nblk % VEC == 0 && p.bins.first_elem[g] % VEC == 0;
        s.vec[g] = vec ? VEC : 1;
        const int64_t nvec = vec ? nblk / VEC : nblk;
        int L = 1;
        while (L < kWave && (nvec + L - 1) / L > kVmax) L <<= 1;
        s.lanes_per_row[g] = L;
        s.tile_begin[g] = tiles;
        const int64_t rpw = kWave / L;
        tiles += (p.bins.rows[g] + rpw - 1) / rpw;
    }
    s.tile_begin[s.nbins] = tiles;
    return s;
}

ProductSchedule spmm_schedule(const darb_plan &p, int64_t B) {
    ProductSchedule s{};
    s.nbins = p.bins.nbins;
    int L = 1;
    while (L < kWave && L < B) L <<= 1;
    s.col_slabs = (B + L - 1) / L;
    int64_t tiles = 0;
    for (int g = 0; g < s.nbins; ++g) {
        s.vec[g] = 1;
        s.lanes_per_row[g] = L;
        s.tile_begin[g] = tiles;
        const int64_t rpw = kWave / L;
        tiles += (p.bins.rows[g] + rpw - 1) / rpw * s.col_slabs;
    }
    s.tile_begin[s.nbins] = tiles;
    return s;
}

template <typename Tw, typename Tx>
hipError_t launch_spmv_t(const darb_plan &p, const void *values, const uint8_t *offsets,
                         const void *x, float *y, hipStream_t st) {
    const ProductSchedule s = spmv_schedule<Tw>(p, values, offsets);
    const int64_t tiles = s.tile_begin[s.nbins];
    const int64_t blocks = (tiles + kWaves - 1) / kWaves;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const Tw *v = static_cast<const Tw *>(values);
    const Tx *xx = static_cast<const Tx *>(x);
    if (p.N <= kLdsMaxFloats) {
        const size_t lds = size_t(p.N) * sizeof(float);
        hipLaunchKernelGGL((spmv_kernel<Tw, Tx, true>), dim3(unsigned(blocks)), dim3(kThreads),
                           lds, st, v, offsets, xx, y, p.d_perm, p.N, p.bins, s);
    } else {
        hipLaunchKernelGGL((spmv_kernel<Tw, Tx, false>), dim3(unsigned(blocks)), dim3(kThreads),
                           0, st, v, offsets, xx, y, p.d_perm, p.N, p.bins, s);
    }
    return hipGetLastError();
}

template <typename Tw, typename Tx>
hipError_t launch_spmm_t(const darb_plan &p, const void *values, const uint8_t *offsets,
                         int64_t B, const void *X, int64_t ldx, float *Y, int64_t ldy,
                         hipStream_t st) {
    const ProductSchedule s = spmm_schedule(p, B);
    const int64_t tiles = s.tile_begin[s.nbins];
    const int64_t blocks = (tiles + kWaves - 1) / kWaves;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((spmm_kernel<Tw, Tx>), dim3(unsigned(blocks)), dim3(kThreads), 0, st,
                       static_cast<const Tw *>(values), offsets, static_cast<const Tx *>(X), ldx,
                       B, Y, ldy, p.d_perm, p.N, p.bins, s);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_spmv(const darb_plan &p, int wdtype, const void *values,
                       const uint8_t *offsets, int xdtype, const void *x, float *y,
                       hipStream_t s) {
    if (wdtype == DARB_F32) return launch_spmv_t<float, float>(p, values, offsets, x, y, s);
    if (xdtype == DARB_F16) return launch_spmv_t<__half, __half>(p, values, offsets, x, y, s);
    return launch_spmv_t<__half, float>(p, values, offsets, x, y, s);
}

hipError_t launch_spmm(const darb_plan &p, int wdtype, const void *values,
                       const uint8_t *offsets, int xdtype, int64_t B, const void *X,
                       int64_t ldx, float *Y, int64_t ldy, hipStream_t s) {
    if (wdtype == DARB_F32)
        return launch_spmm_t<float, float>(p, values, offsets, B, X, ldx, Y, ldy, s);
    if (xdtype == DARB_F16)
        return launch_spmm_t<__half, __half>(p, values, offsets, B, X, ldx, Y, ldy, s);
    return launch_spmm_t<__half, float>(p, values, offsets, B, X, ldx, Y, ldy, s);
}

}  // namespace darb
