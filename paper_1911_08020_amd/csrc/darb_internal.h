// Internal declarations shared by the host code and the kernel launchers of
// the DARB library.  Not part of the public ABI (include/darb.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "darb.h"

namespace darb {

constexpr int kMaxBins = 8;      // block sizes 1, 2, ..., 128
constexpr int kMaxLog2B = 7;
constexpr int kWave = 64;        // CDNA wavefront width

// The block-size groups, passed to kernels by value.
struct BinTable {
    int32_t nbins;
    int32_t log2b[kMaxBins];
    int64_t first_row[kMaxBins];   // storage-order index of the group's first row
    int64_t rows[kMaxBins];
    int64_t first_elem[kMaxBins];  // slot of the group's first retained weight
    int64_t nblk[kMaxBins];        // retained weights per row
    int64_t first_word[kMaxBins];  // packed offsets: the group's first 32-bit word
};

// Per-launch work split of the product kernels.  Every workgroup belongs to one
// block-size group g: blocks [block_begin[g], block_begin[g+1]).
struct ProductSchedule {
    int32_t nbins;
    int32_t block_begin[kMaxBins + 1];
    int32_t log2_lanes[kMaxBins];     // log2 of the lanes that share one row
    int32_t vec[kMaxBins];            // SpMV: elements per vector load (1 = scalar path)
    int32_t ksplit[kMaxBins];         // SpMM: waves that split one row group's weights
    int32_t col_slabs;                // SpMM: batch-column slabs per row block
    int32_t stage_loads;              // SpMV: 16-byte loads per thread to stage x
};

}  // namespace darb

struct darb_plan {
    int64_t M = 0, N = 0, nnz = 0;
    int mode = 0, b_min = 1, b_max = 1;
    std::vector<uint8_t> log2b;
    std::vector<int64_t> row_start;
    std::vector<int32_t> perm;
    darb::BinTable bins{};
    int64_t workspace_bytes = 0;
    int64_t packed_words = 0;       // 32-bit words of the bit-packed offsets
    // device side (inside the caller's workspace)
    int32_t *d_perm = nullptr;      // [M] original row stored i-th
    int64_t *d_rowinfo = nullptr;   // [M] (row_start[r] << 8) | log2b[r], original order
    int device = -1;
    int cus = 0;                    // compute units of that device
    bool device_built = false;      // built on the device: the host vectors are empty
};

namespace darb {

// error reporting (thread-local detail string)
int fail(int code, const std::string &detail);
void clear_error();

// kernel launchers (return hipError_t of the launch)
hipError_t launch_encode(const darb_plan &p, int wdtype, const void *W, int64_t ldw,
                         void *values, uint8_t *offsets, hipStream_t s);
hipError_t launch_decode(const darb_plan &p, int wdtype, const void *values,
                         const uint8_t *offsets, void *W_out, int64_t ldw, hipStream_t s);
// The products read the offsets from exactly one of `offsets` (one byte per
// retained weight) and `packed` (log2 b bits per retained weight); the other is NULL.
hipError_t launch_spmv(const darb_plan &p, int wdtype, const void *values,
                       const uint8_t *offsets, const uint32_t *packed, int xdtype,
                       const void *x, float *y, hipStream_t s);
hipError_t launch_spmm(const darb_plan &p, int wdtype, const void *values,
                       const uint8_t *offsets, const uint32_t *packed, int xdtype, int64_t B,
                       const void *X, int64_t ldx, float *Y, int64_t ldy, hipStream_t s);
// INT8 values: per-row codes and scales, and the products on them (scales indexed
// by original row, applied to each row's fp32 sum).
hipError_t launch_quantize_i8(const darb_plan &p, int wdtype, const void *values, int8_t *codes,
                              float *scales, hipStream_t s);
hipError_t launch_spmv_i8(const darb_plan &p, const int8_t *codes, const float *scales,
                          const uint8_t *offsets, const uint32_t *packed, int xdtype,
                          const void *x, float *y, hipStream_t s);
hipError_t launch_spmm_i8(const darb_plan &p, const int8_t *codes, const float *scales,
                          const uint8_t *offsets, const uint32_t *packed, int xdtype, int64_t B,
                          const void *X, int64_t ldx, float *Y, int64_t ldy, hipStream_t s);
hipError_t launch_pack_offsets(const darb_plan &p, const uint8_t *offsets, uint32_t *packed,
                               hipStream_t s);
hipError_t launch_unpack_offsets(const darb_plan &p, const uint32_t *packed, uint8_t *offsets,
                                 hipStream_t s);
int64_t prune_workspace_bytes(int64_t M, int64_t N, int wdtype);
hipError_t launch_prune_counts(int64_t M, int64_t N, int wdtype, const void *W, int64_t ldw,
                               int64_t k, int64_t *counts, void *workspace, hipStream_t s);
// the same with the workspace in the library's fixed per-device array (no allocation);
// M must be at most prune_static_max_rows()
int64_t prune_static_max_rows();
hipError_t launch_prune_counts_static(int64_t M, int64_t N, int wdtype, const void *W,
                                      int64_t ldw, int64_t k, int64_t *counts, hipStream_t s);
// One fused LSTM step (recurrent product and gate cell of every hidden unit), when
// lstm_step_fusable: h_in is read, h_out written (distinct buffers).
bool lstm_step_fusable(const darb_plan &whh, int64_t batch, const float *h, const float *h2);
hipError_t launch_lstm_step(const darb_plan &whh, int wdtype, const void *values,
                            const uint8_t *offsets, int64_t H, int64_t batch, const float *h_in,
                            const float *U, int64_t ldu, float *c, float *h_out, float *h_seq,
                            int64_t ld_seq, hipStream_t s);
hipError_t launch_lstm_cell(int64_t H, int64_t batch, const float *G, const float *U,
                            int64_t ldu, float *h, float *c, float *h_seq, int64_t ld_seq,
                            hipStream_t s);
// The plan's storage order and per-row table from device-side kept counts, and the
// group summary (rows, first_row, first_elem, first_word: 8 int64 each) at the start
// of `scratch` (plan_device_scratch_bytes(M), 256-byte aligned).
int64_t plan_device_scratch_bytes(int64_t M);
hipError_t launch_plan_device(int64_t M, int64_t N, const int64_t *counts, int64_t kept, int mode,
                              int lmin, int lmax, int32_t *perm, int64_t *rowinfo, void *scratch,
                              hipStream_t s);
hipError_t launch_stream_read(const void *buf, int64_t bytes, float *sink, hipStream_t s);
hipError_t launch_stream_read_shape(const void *buf, int64_t bytes, int threads, int vectors,
                                   float *sink, hipStream_t s);
hipError_t launch_stream_copy(void *dst, const void *src, int64_t bytes, hipStream_t s);

}  // namespace darb
