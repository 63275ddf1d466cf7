// Conversion between the one-byte offsets the encode writes and the bit-packed
// offsets of section 4.2 (log2 b bits per retained weight; the layout is
// described in packed_bits.h).
#include "darb_internal.h"
#include "packed_bits.h"

namespace darb {
namespace {

constexpr int kThreads = 256;

// Group of a global index: the last group whose first index is <= i (groups are
// in ascending order; a group of b = 1 owns no words, and the group after it
// starts at the same word, so "last" picks the owner).  Unrolled selects keep the
// table in scalar registers.
__device__ __forceinline__ int owning_group(const int64_t (&first)[kMaxBins], int nbins,
                                            int64_t i) {
    int g = 0;
#pragma unroll
    for (int b = 1; b < kMaxBins; ++b) g = (b < nbins && first[b] <= i) ? b : g;
    return g;
}

template <typename T>
__device__ __forceinline__ T pick(const T (&a)[kMaxBins], int g) {
    T r = a[0];
#pragma unroll
    for (int b = 1; b < kMaxBins; ++b) r = (b == g) ? a[b] : r;
    return r;
}

// One thread per packed word.  Word w of a run covers bits [32w, 32w + 32) of the
// run's bit string; the indices that touch it are those of weights
// floor(32w / l) ... floor((32w + 31) / l) of the run.
__global__ __launch_bounds__(kThreads) void pack_kernel(const uint8_t *__restrict__ offsets,
                                                        uint32_t *__restrict__ packed,
                                                        int64_t words, BinTable bins) {
    const int64_t wi = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (wi >= words) return;
    const int g = owning_group(bins.first_word, bins.nbins, wi);
    const int l = pick(bins.log2b, g);                   // >= 1: this group has words
    const int64_t wg = wi - pick(bins.first_word, g);
    const int64_t run = wg / l;
    const int w = int(wg - run * l);
    const int64_t count = pick(bins.rows, g) * pick(bins.nblk, g);
    const int64_t left = count - run * 32;               // weights in this run (>= 1)
    const uint8_t *src = offsets + pick(bins.first_elem, g) + run * 32;
    const uint32_t mask = (1u << l) - 1u;
    const int s_lo = (32 * w) / l;
    int s_hi = (32 * w + 31) / l;
    if (s_hi > 31) s_hi = 31;
    if (s_hi > left - 1) s_hi = int(left - 1);
    uint32_t word = 0;
    for (int s = s_lo; s <= s_hi; ++s) {
        const uint32_t off = uint32_t(src[s]) & mask;
        const int p = s * l - 32 * w;                    // in (-l, 32)
        word |= p >= 0 ? off << p : off >> (-p);
    }
    packed[wi] = word;
}

// One thread per retained weight.
__global__ __launch_bounds__(kThreads) void unpack_kernel(const uint32_t *__restrict__ packed,
                                                          uint8_t *__restrict__ offsets,
                                                          int64_t nnz, BinTable bins) {
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= nnz) return;
    const int g = owning_group(bins.first_elem, bins.nbins, i);
    const int l = pick(bins.log2b, g);
    if (l == 0) {                                        // b = 1: no words, index 0
        offsets[i] = 0;
        return;
    }
    const PackedGroup pg = packed_group(packed, pick(bins.first_word, g), l);
    const int64_t j = i - pick(bins.first_elem, g);
    offsets[i] = uint8_t(packed_bits32(packed_load2(pg, j)) & pg.mask);
}

}  // namespace

hipError_t launch_pack_offsets(const darb_plan &p, const uint8_t *offsets, uint32_t *packed,
                               hipStream_t s) {
    if (p.packed_words == 0) return hipSuccess;
    const int64_t blocks = (p.packed_words + kThreads - 1) / kThreads;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(pack_kernel, dim3(unsigned(blocks)), dim3(kThreads), 0, s, offsets, packed,
                       p.packed_words, p.bins);
    return hipGetLastError();
}

hipError_t launch_unpack_offsets(const darb_plan &p, const uint32_t *packed, uint8_t *offsets,
                                 hipStream_t s) {
    const int64_t blocks = (p.nnz + kThreads - 1) / kThreads;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(unpack_kernel, dim3(unsigned(blocks)), dim3(kThreads), 0, s, packed,
                       offsets, p.nnz, p.bins);
    return hipGetLastError();
}

}  // namespace darb
