// Decode to the masked dense matrix, the LSTM cell of the recurrent workload,
// and the HBM stream kernels the DARB kernels are measured against.
#include "darb_internal.h"
#include "lstm_cell.h"

namespace darb {
namespace {

constexpr int kThreads = 256;

// One thread per (storage-order row, column): the column's block k = c >> log2b
// keeps column k*b + off[k]; every other column of the row is +0.0.
template <typename Bits>
__global__ __launch_bounds__(kThreads) void decode_kernel(
    const Bits *__restrict__ values, const uint8_t *__restrict__ offsets, Bits *__restrict__ W,
    int64_t ldw, int64_t N, const int32_t *__restrict__ perm, BinTable bins, int64_t col_blocks) {
    const int64_t i = blockIdx.x / col_blocks;
    const int64_t c = (blockIdx.x - i * col_blocks) * int64_t(kThreads) + threadIdx.x;
    if (c >= N) return;
    int g = 0;
    while (g + 1 < bins.nbins && i >= bins.first_row[g + 1]) ++g;
    const int lb = bins.log2b[g];
    const int64_t e = bins.first_elem[g] + (i - bins.first_row[g]) * bins.nblk[g] + (c >> lb);
    const int64_t j = c & ((int64_t(1) << lb) - 1);
    W[int64_t(perm[i]) * ldw + c] = (offsets[e] == j) ? values[e] : Bits(0);
}

// gates = G + U (G: recurrent product [4H x batch], U: input product slice of
// this step, leading dimension ldu), gate order (i, f, g, o).
__global__ __launch_bounds__(kThreads) void lstm_cell_kernel(
    int64_t H, int64_t batch, const float *__restrict__ G, const float *__restrict__ U,
    int64_t ldu, float *__restrict__ h, float *__restrict__ c, float *__restrict__ h_seq,
    int64_t ld_seq) {
    const int64_t idx = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (idx >= H * batch) return;
    const int64_t u = idx / batch, n = idx - u * batch;
    const float gi = G[u * batch + n] + U[u * ldu + n];
    const float gf = G[(H + u) * batch + n] + U[(H + u) * ldu + n];
    const float gg = G[(2 * H + u) * batch + n] + U[(2 * H + u) * ldu + n];
    const float go = G[(3 * H + u) * batch + n] + U[(3 * H + u) * ldu + n];
    float cn = c[idx];
    const float hn = lstm_cell(gi, gf, gg, go, cn);
    c[idx] = cn;
    h[idx] = hn;
    h_seq[u * ld_seq + n] = hn;
}

constexpr int kStreamBlocks = 8192;
constexpr int kReadUnroll = 4;     // 16-byte loads in flight per thread

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Each workgroup reads one contiguous chunk of kReadUnroll * kThreads 16-byte
// vectors with non-temporal loads, all issued before they are summed; one float per
// workgroup goes to sink[blockIdx.x % kStreamBlocks] so the loads are kept.
__global__ __launch_bounds__(kThreads) void stream_read_kernel(const f32x4 *__restrict__ buf,
                                                               int64_t n16, float *sink) {
    const int64_t base = int64_t(blockIdx.x) * (kReadUnroll * kThreads) + threadIdx.x;
    f32x4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) {
        const int64_t i = base + int64_t(u) * kThreads;
        v[u] = __builtin_nontemporal_load(buf + (i < n16 ? i : n16 - 1));
    }
    float s = 0.0f;
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) s += (v[u][0] + v[u][1]) + (v[u][2] + v[u][3]);
    __shared__ float part[kThreads / 64];
    for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x / 64] = s;
    __syncthreads();
    if (threadIdx.x == 0)
        sink[blockIdx.x % kStreamBlocks] = (part[0] + part[1]) + (part[2] + part[3]);
}

// The same read in other launch shapes: THREADS threads per workgroup, each issuing
// VPL 16-byte non-temporal loads (lanes interleaved, so every load instruction of a
// wave covers 1 KiB) before summing them.  The sum goes to memory only when it
// equals a value no real data produces, so the loads cannot be elided and nothing is
// normally written: the launch measures the read alone.
template <int THREADS, int VPL>
__global__ __launch_bounds__(THREADS) void stream_read_shape_kernel(
    const f32x4 *__restrict__ buf, int64_t n16, float *sink) {
    const int64_t base = int64_t(blockIdx.x) * (VPL * THREADS) + threadIdx.x;
    f32x4 v[VPL];
#pragma unroll
    for (int u = 0; u < VPL; ++u) {
        const int64_t i = base + int64_t(u) * THREADS;
        v[u] = __builtin_nontemporal_load(buf + (i < n16 ? i : n16 - 1));
    }
    float s = 0.0f;
#pragma unroll
    for (int u = 0; u < VPL; ++u) s += (v[u][0] + v[u][1]) + (v[u][2] + v[u][3]);
    if (s == -0x1.5p-126f) sink[blockIdx.x % kStreamBlocks] = s;
}

__global__ __launch_bounds__(kThreads) void stream_copy_kernel(float4 *__restrict__ dst,
                                                               const float4 *__restrict__ src,
                                                               int64_t n16) {
    for (int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x; i < n16;
         i += int64_t(gridDim.x) * kThreads)
        dst[i] = src[i];
}

template <typename Bits>
hipError_t launch_decode_t(const darb_plan &p, const void *values, const uint8_t *offsets,
                           void *W, int64_t ldw, hipStream_t s) {
    const int64_t col_blocks = (p.N + kThreads - 1) / kThreads;
    const int64_t blocks = p.M * col_blocks;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((decode_kernel<Bits>), dim3(unsigned(blocks)), dim3(kThreads), 0, s,
                       static_cast<const Bits *>(values), offsets, static_cast<Bits *>(W), ldw,
                       p.N, p.d_perm, p.bins, col_blocks);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const darb_plan &p, int wdtype, const void *values,
                         const uint8_t *offsets, void *W_out, int64_t ldw, hipStream_t s) {
    if (wdtype == DARB_F32) return launch_decode_t<uint32_t>(p, values, offsets, W_out, ldw, s);
    return launch_decode_t<uint16_t>(p, values, offsets, W_out, ldw, s);
}

hipError_t launch_lstm_cell(int64_t H, int64_t batch, const float *G, const float *U,
                            int64_t ldu, float *h, float *c, float *h_seq, int64_t ld_seq,
                            hipStream_t s) {
    const int64_t n = H * batch;
    const int64_t blocks = (n + kThreads - 1) / kThreads;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(lstm_cell_kernel, dim3(unsigned(blocks)), dim3(kThreads), 0, s, H, batch,
                       G, U, ldu, h, c, h_seq, ld_seq);
    return hipGetLastError();
}

hipError_t launch_stream_read(const void *buf, int64_t bytes, float *sink, hipStream_t s) {
    const int64_t n16 = bytes / 16;
    const int64_t blocks = (n16 + kReadUnroll * kThreads - 1) / (kReadUnroll * kThreads);
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(stream_read_kernel, dim3(unsigned(blocks)), dim3(kThreads), 0, s,
                       static_cast<const f32x4 *>(buf), n16, sink);
    return hipGetLastError();
}

hipError_t launch_stream_read_shape(const void *buf, int64_t bytes, int threads, int vectors,
                                   float *sink, hipStream_t s) {
    const int64_t n16 = bytes / 16;
    const int64_t per_block = int64_t(threads) * vectors;
    const int64_t blocks = (n16 + per_block - 1) / per_block;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const f32x4 *b = static_cast<const f32x4 *>(buf);
#define DARB_READ_SHAPE(T, V)                                                               \
    if (threads == T && vectors == V) {                                                     \
        hipLaunchKernelGGL((stream_read_shape_kernel<T, V>), dim3(unsigned(blocks)), dim3(T), \
                           0, s, b, n16, sink);                                             \
        return hipGetLastError();                                                           \
    }
    DARB_READ_SHAPE(64, 4) DARB_READ_SHAPE(64, 8) DARB_READ_SHAPE(128, 4)
    DARB_READ_SHAPE(256, 1) DARB_READ_SHAPE(256, 2) DARB_READ_SHAPE(256, 4) DARB_READ_SHAPE(256, 8)
    DARB_READ_SHAPE(512, 1) DARB_READ_SHAPE(512, 2) DARB_READ_SHAPE(512, 4)
    DARB_READ_SHAPE(1024, 1) DARB_READ_SHAPE(1024, 2) DARB_READ_SHAPE(1024, 4)
#undef DARB_READ_SHAPE
    return hipErrorInvalidValue;
}

hipError_t launch_stream_copy(void *dst, const void *src, int64_t bytes, hipStream_t s) {
    const int64_t n16 = bytes / 16;
    int64_t blocks = (n16 + kThreads - 1) / kThreads;
    if (blocks > kStreamBlocks) blocks = kStreamBlocks;
    hipLaunchKernelGGL(stream_copy_kernel, dim3(unsigned(blocks)), dim3(kThreads), 0, s,
                       static_cast<float4 *>(dst), static_cast<const float4 *>(src), n16);
    return hipGetLastError();
}

}  // namespace darb
