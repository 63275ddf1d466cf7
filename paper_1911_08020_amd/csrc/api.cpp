// Host side of the DARB library: plan construction (section 3.2 block-size
// rule and grouped layout), argument checking and dispatch to the kernels.
#include <cmath>
#include <cstring>
#include <new>
#include <string>

#include "darb_internal.h"

namespace darb {

static thread_local std::string g_last_error;

int fail(int code, const std::string &detail) {
    g_last_error = detail;
    return code;
}

void clear_error() { g_last_error.clear(); }

static bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

static constexpr int64_t kMaxColumns = (int64_t(1) << 31) - 256;

// workspace layout: perm (int32 [M]) padded to 256 bytes, then rowinfo (int64 [M])
static int64_t perm_bytes(int64_t M) { return (M * int64_t(sizeof(int32_t)) + 255) / 256 * 256; }

static int log2_exact(int64_t v) {
    int l = 0;
    while ((int64_t(1) << l) != v) ++l;
    return l;
}

// Section 3.2: move the row density d to a power-of-two fraction and take its
// reciprocal.  With d = m * 2^e (frexp, m in [0.5, 1)), the smallest power-of-
// two fraction >= d is 2^(e-1) when m == 0.5 (d already is one) and 2^e
// otherwise; the largest one <= d is 2^(e-1).  Rounding up therefore gives
// log2 b = 1 - e (m == 0.5) or -e, rounding down gives 1 - e.  Paper mode rounds
// up for d >= D and down for d < D; floor mode always rounds up.  A row of
// density 0 gets b_max.  The result is clamped to [log2 b_min, log2 b_max].
static int row_log2b(double d, double D, int mode, int lmin, int lmax) {
    if (d == 0.0) return lmax;
    int e = 0;
    const double m = std::frexp(d, &e);
    const bool exact = (m == 0.5);
    const bool round_up = (mode == DARB_ROUND_FLOOR) || (d >= D);
    int64_t l = (round_up && !exact) ? -int64_t(e) : 1 - int64_t(e);
    if (l < lmin) l = lmin;
    if (l > lmax) l = lmax;
    return int(l);
}

}  // namespace darb

using namespace darb;

extern "C" {

int darb_version(void) { return 300; }

const char *darb_strerror(int code) {
    switch (code) {
        case DARB_OK: return "success";
        case DARB_E_INVALID: return "invalid argument";
        case DARB_E_DTYPE: return "unsupported dtype";
        case DARB_E_NOT_UPLOADED: return "plan has no device metadata (call darb_plan_upload)";
        case DARB_E_HIP: return "HIP runtime error";
        case DARB_E_NOMEM: return "host allocation failed";
        case DARB_E_WORKSPACE: return "workspace too small";
        default: return "unknown error code";
    }
}

const char *darb_last_error(void) { return g_last_error.c_str(); }

int darb_plan_create_counts(int64_t M, int64_t N, const int64_t *row_count, int64_t kept,
                            int round_mode, int b_min, int b_max, darb_plan **out) {
    clear_error();
    if (!out) return fail(DARB_E_INVALID, "out is NULL");
    *out = nullptr;
    if (M < 1 || M >= (int64_t(1) << 31)) return fail(DARB_E_INVALID, "M must be in [1, 2^31)");
    if (N < 1 || N > kMaxColumns)
        return fail(DARB_E_INVALID, "N must be in [1, 2^31 - 256]");
    if (!row_count) return fail(DARB_E_INVALID, "row_count is NULL");
    if (kept < 0 || kept > M * N) return fail(DARB_E_INVALID, "kept must be in [0, M*N]");
    std::vector<double> d;
    try {
        d.resize(M);
    } catch (const std::bad_alloc &) {
        return fail(DARB_E_NOMEM, "densities");
    }
    for (int64_t r = 0; r < M; ++r) {
        if (row_count[r] < 0 || row_count[r] > N)
            return fail(DARB_E_INVALID, "row_count[" + std::to_string(r) + "] not in [0, N]");
        d[r] = double(row_count[r]) / double(N);
    }
    return darb_plan_create(M, N, d.data(), double(kept) / (double(M) * double(N)), round_mode,
                            b_min, b_max, out);
}

int darb_plan_create(int64_t M, int64_t N, const double *row_density, double matrix_density,
                     int round_mode, int b_min, int b_max, darb_plan **out) {
    clear_error();
    if (!out) return fail(DARB_E_INVALID, "out is NULL");
    *out = nullptr;
    if (M < 1 || M >= (int64_t(1) << 31)) return fail(DARB_E_INVALID, "M must be in [1, 2^31)");
    // the products form a column as (block << log2 b) + offset in 32 bits
    if (N < 1 || N > kMaxColumns)
        return fail(DARB_E_INVALID, "N must be in [1, 2^31 - 256]");
    if (!row_density) return fail(DARB_E_INVALID, "row_density is NULL");
    if (round_mode != DARB_ROUND_FLOOR && round_mode != DARB_ROUND_PAPER)
        return fail(DARB_E_INVALID, "unknown round_mode");
    if (!is_pow2(b_min) || !is_pow2(b_max) || b_min > b_max || b_max > 128)
        return fail(DARB_E_INVALID, "b_min, b_max must be powers of two, 1 <= b_min <= b_max <= 128");
    if (!(matrix_density >= 0.0 && matrix_density <= 1.0))
        return fail(DARB_E_INVALID, "matrix_density must be in [0, 1]");
    for (int64_t r = 0; r < M; ++r) {
        const double d = row_density[r];
        if (!(d >= 0.0 && d <= 1.0))
            return fail(DARB_E_INVALID, "row_density[" + std::to_string(r) + "] not in [0, 1]");
    }
    darb_plan *p = new (std::nothrow) darb_plan();
    if (!p) return fail(DARB_E_NOMEM, "plan allocation");
    try {
        p->M = M;
        p->N = N;
        p->mode = round_mode;
        p->b_min = b_min;
        p->b_max = b_max;
        p->log2b.resize(M);
        p->row_start.resize(M);
        p->perm.resize(M);
    } catch (const std::bad_alloc &) {
        delete p;
        return fail(DARB_E_NOMEM, "plan arrays");
    }
    const int lmin = log2_exact(b_min), lmax = log2_exact(b_max);
    int64_t count[kMaxBins] = {0};
    for (int64_t r = 0; r < M; ++r) {
        const int l = row_log2b(row_density[r], matrix_density, round_mode, lmin, lmax);
        p->log2b[r] = uint8_t(l);
        ++count[l];
    }
    // grouped layout: groups by ascending block size, rows ascending inside
    int64_t group_row[kMaxBins], group_elem[kMaxBins];
    int64_t row = 0, elem = 0, words = 0;
    BinTable &bt = p->bins;
    bt.nbins = 0;
    for (int l = 0; l <= kMaxLog2B; ++l) {
        const int64_t nblk = (N + (int64_t(1) << l) - 1) >> l;
        group_row[l] = row;
        group_elem[l] = elem;
        if (count[l] > 0) {
            const int g = bt.nbins++;
            bt.log2b[g] = l;
            bt.first_row[g] = row;
            bt.rows[g] = count[l];
            bt.first_elem[g] = elem;
            bt.nblk[g] = nblk;
            bt.first_word[g] = words;
        }
        row += count[l];
        elem += count[l] * nblk;
        // packed offsets (section 4.2): runs of 32 weights, log2 b words per run
        words += (count[l] * nblk + 31) / 32 * l;
    }
    // the per-row table packs a slot index and log2 b into 64 bits (slot << 8)
    if (elem >= (int64_t(1) << 55)) {
        delete p;
        return fail(DARB_E_INVALID, "more than 2^55 retained weights");
    }
    p->nnz = elem;
    p->packed_words = words;
    for (int64_t r = 0; r < M; ++r) {
        const int l = p->log2b[r];
        const int64_t nblk = (N + (int64_t(1) << l) - 1) >> l;
        const int64_t i = group_row[l]++;
        p->perm[i] = int32_t(r);
        p->row_start[r] = group_elem[l];
        group_elem[l] += nblk;
    }
    p->workspace_bytes = perm_bytes(M) + M * int64_t(sizeof(int64_t));
    *out = p;
    return DARB_OK;
}

int darb_plan_info(const darb_plan *p, darb_plan_info_t *info) {
    clear_error();
    if (!p || !info) return fail(DARB_E_INVALID, "NULL argument");
    std::memset(info, 0, sizeof(*info));
    info->M = p->M;
    info->N = p->N;
    info->nnz = p->nnz;
    info->workspace_bytes = p->workspace_bytes;
    info->packed_words = p->packed_words;
    info->nbins = p->bins.nbins;
    for (int g = 0; g < p->bins.nbins; ++g) {
        info->bins[g].log2b = p->bins.log2b[g];
        info->bins[g].first_row = p->bins.first_row[g];
        info->bins[g].rows = p->bins.rows[g];
        info->bins[g].first_elem = p->bins.first_elem[g];
        info->bins[g].nblk = p->bins.nblk[g];
        info->bins[g].first_word = p->bins.first_word[g];
    }
    return DARB_OK;
}

int darb_plan_export(const darb_plan *p, uint8_t *log2b, int64_t *row_start, int32_t *perm) {
    clear_error();
    if (!p) return fail(DARB_E_INVALID, "plan is NULL");
    if (p->device_built) {
        // the tables live only in the build workspace: copy them back
        std::vector<int64_t> rowinfo;
        try {
            rowinfo.resize(p->M);
        } catch (const std::bad_alloc &) {
            return fail(DARB_E_NOMEM, "rowinfo");
        }
        hipError_t e = hipMemcpy(rowinfo.data(), p->d_rowinfo, p->M * sizeof(int64_t),
                                 hipMemcpyDeviceToHost);
        if (e == hipSuccess && perm)
            e = hipMemcpy(perm, p->d_perm, p->M * sizeof(int32_t), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return fail(DARB_E_HIP, std::string("plan export: ") + hipGetErrorString(e));
        for (int64_t r = 0; r < p->M; ++r) {
            if (log2b) log2b[r] = uint8_t(rowinfo[r] & 0xFF);
            if (row_start) row_start[r] = rowinfo[r] >> 8;
        }
        return DARB_OK;
    }
    if (log2b) std::memcpy(log2b, p->log2b.data(), p->M * sizeof(uint8_t));
    if (row_start) std::memcpy(row_start, p->row_start.data(), p->M * sizeof(int64_t));
    if (perm) std::memcpy(perm, p->perm.data(), p->M * sizeof(int32_t));
    return DARB_OK;
}

int darb_plan_upload(darb_plan *p, void *workspace, int64_t workspace_bytes, void *stream) {
    clear_error();
    if (!p || !workspace) return fail(DARB_E_INVALID, "NULL argument");
    if (p->device_built)
        return fail(DARB_E_INVALID, "a plan built on the device stays in its build workspace");
    if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0)
        return fail(DARB_E_INVALID, "workspace must be 256-byte aligned");
    if (workspace_bytes < p->workspace_bytes)
        return fail(DARB_E_WORKSPACE, "workspace needs " + std::to_string(p->workspace_bytes) +
                                          " bytes, got " + std::to_string(workspace_bytes));
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(DARB_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    std::vector<int64_t> rowinfo;
    try {
        rowinfo.resize(p->M);
    } catch (const std::bad_alloc &) {
        return fail(DARB_E_NOMEM, "rowinfo");
    }
    for (int64_t r = 0; r < p->M; ++r) rowinfo[r] = (p->row_start[r] << 8) | p->log2b[r];
    int32_t *d_perm = static_cast<int32_t *>(workspace);
    int64_t *d_rowinfo = reinterpret_cast<int64_t *>(static_cast<char *>(workspace) +
                                                     perm_bytes(p->M));
    hipStream_t s = static_cast<hipStream_t>(stream);
    e = hipMemcpyAsync(d_perm, p->perm.data(), p->M * sizeof(int32_t), hipMemcpyHostToDevice, s);
    if (e == hipSuccess)
        e = hipMemcpyAsync(d_rowinfo, rowinfo.data(), p->M * sizeof(int64_t),
                           hipMemcpyHostToDevice, s);
    // the host vector dies on return: make sure the copies have consumed it
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(DARB_E_HIP, std::string("plan upload: ") + hipGetErrorString(e));
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return fail(DARB_E_HIP, std::string("device attribute: ") + hipGetErrorString(e));
    p->d_perm = d_perm;
    p->d_rowinfo = d_rowinfo;
    p->device = dev;
    p->cus = cus;
    return DARB_OK;
}

void darb_plan_destroy(darb_plan *p) { delete p; }

static int64_t device_plan_bytes(int64_t M) {
    return perm_bytes(M) + (M * int64_t(sizeof(int64_t)) + 255) / 256 * 256 +
           plan_device_scratch_bytes(M);
}

int darb_plan_device_workspace(int64_t M, int64_t *bytes) {
    clear_error();
    if (!bytes || M < 1 || M >= (int64_t(1) << 31))
        return fail(DARB_E_INVALID, "bytes is NULL or M not in [1, 2^31)");
    *bytes = device_plan_bytes(M);
    return DARB_OK;
}

int darb_plan_create_device(int64_t M, int64_t N, const int64_t *row_count, int64_t kept,
                            int round_mode, int b_min, int b_max, void *workspace,
                            int64_t workspace_bytes, void *stream, darb_plan **out) {
    clear_error();
    if (!out) return fail(DARB_E_INVALID, "out is NULL");
    *out = nullptr;
    if (M < 1 || M >= (int64_t(1) << 31)) return fail(DARB_E_INVALID, "M must be in [1, 2^31)");
    if (N < 1 || N > kMaxColumns) return fail(DARB_E_INVALID, "N must be in [1, 2^31 - 256]");
    if (!row_count || !workspace) return fail(DARB_E_INVALID, "NULL buffer");
    if ((reinterpret_cast<uintptr_t>(row_count) & 7) != 0)
        return fail(DARB_E_INVALID, "row_count must be 8-byte aligned");
    if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0)
        return fail(DARB_E_INVALID, "workspace must be 256-byte aligned");
    if (kept < 0 || kept > M * N) return fail(DARB_E_INVALID, "kept must be in [0, M*N]");
    if (round_mode != DARB_ROUND_FLOOR && round_mode != DARB_ROUND_PAPER)
        return fail(DARB_E_INVALID, "unknown round_mode");
    if (!is_pow2(b_min) || !is_pow2(b_max) || b_min > b_max || b_max > 128)
        return fail(DARB_E_INVALID, "b_min, b_max must be powers of two, 1 <= b_min <= b_max <= 128");
    const int64_t need = device_plan_bytes(M);
    if (workspace_bytes < need)
        return fail(DARB_E_WORKSPACE, "device plan needs " + std::to_string(need) + " bytes, got " +
                                          std::to_string(workspace_bytes));
    int dev = -1, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return fail(DARB_E_HIP, std::string("device: ") + hipGetErrorString(e));
    char *base = static_cast<char *>(workspace);
    int32_t *d_perm = reinterpret_cast<int32_t *>(base);
    int64_t *d_rowinfo = reinterpret_cast<int64_t *>(base + perm_bytes(M));
    void *scratch = base + perm_bytes(M) + (M * int64_t(sizeof(int64_t)) + 255) / 256 * 256;
    hipStream_t s = static_cast<hipStream_t>(stream);
    e = launch_plan_device(M, N, row_count, kept, round_mode, log2_exact(b_min), log2_exact(b_max),
                           d_perm, d_rowinfo, scratch, s);
    int64_t summary[4 * kMaxBins];
    if (e == hipSuccess)
        e = hipMemcpyAsync(summary, scratch, sizeof(summary), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(DARB_E_HIP, std::string("device plan: ") + hipGetErrorString(e));
    darb_plan *p = new (std::nothrow) darb_plan();
    if (!p) return fail(DARB_E_NOMEM, "plan allocation");
    p->M = M;
    p->N = N;
    p->mode = round_mode;
    p->b_min = b_min;
    p->b_max = b_max;
    BinTable &bt = p->bins;
    bt.nbins = 0;
    int64_t elem = 0, words = 0;
    for (int l = 0; l <= kMaxLog2B; ++l) {
        const int64_t rows = summary[l];
        const int64_t nblk = (N + (int64_t(1) << l) - 1) >> l;
        if (rows > 0) {
            const int g = bt.nbins++;
            bt.log2b[g] = l;
            bt.first_row[g] = summary[kMaxBins + l];
            bt.rows[g] = rows;
            bt.first_elem[g] = summary[2 * kMaxBins + l];
            bt.nblk[g] = nblk;
            bt.first_word[g] = summary[3 * kMaxBins + l];
        }
        elem += rows * nblk;
        words += (rows * nblk + 31) / 32 * l;
    }
    if (elem >= (int64_t(1) << 55)) {
        delete p;
        return fail(DARB_E_INVALID, "more than 2^55 retained weights");
    }
    p->nnz = elem;
    p->packed_words = words;
    p->workspace_bytes = need;
    p->d_perm = d_perm;
    p->d_rowinfo = d_rowinfo;
    p->device = dev;
    p->cus = cus;
    p->device_built = true;
    *out = p;
    return DARB_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// device entry points
// ---------------------------------------------------------------------------

static int check_uploaded(const darb_plan *p) {
    if (!p) return fail(DARB_E_INVALID, "plan is NULL");
    if (!p->d_perm) return fail(DARB_E_NOT_UPLOADED, "plan was not uploaded");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(DARB_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    if (dev != p->device)
        return fail(DARB_E_INVALID, "plan was uploaded on device " + std::to_string(p->device) +
                                        ", current device is " + std::to_string(dev));
    return DARB_OK;
}

static bool valid_dtype(int t) { return t == DARB_F32 || t == DARB_F16; }

static int launched(hipError_t e, const char *what) {
    if (e == hipSuccess) e = hipGetLastError();
    else (void)hipGetLastError();
    if (e != hipSuccess) return fail(DARB_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
    return DARB_OK;
}

static int check_product_dtypes(int wdtype, int xdtype) {
    if (!valid_dtype(wdtype) || !valid_dtype(xdtype)) return fail(DARB_E_DTYPE, "unknown dtype");
    if (wdtype == DARB_F32 && xdtype != DARB_F32)
        return fail(DARB_E_DTYPE, "fp32 weights need fp32 activations");
    return DARB_OK;
}

extern "C" {

int darb_encode(const darb_plan *p, int wdtype, const void *W, int64_t ldw, void *values,
                uint8_t *offsets, void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    if (!valid_dtype(wdtype)) return fail(DARB_E_DTYPE, "unknown weight dtype");
    if (!W || !values || !offsets) return fail(DARB_E_INVALID, "NULL buffer");
    if (ldw < p->N) return fail(DARB_E_INVALID, "ldw < N");
    return launched(launch_encode(*p, wdtype, W, ldw, values, offsets,
                                  static_cast<hipStream_t>(stream)), "encode launch");
}

int darb_decode(const darb_plan *p, int wdtype, const void *values, const uint8_t *offsets,
                void *W_out, int64_t ldw, void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    if (!valid_dtype(wdtype)) return fail(DARB_E_DTYPE, "unknown weight dtype");
    if (!W_out || !values || !offsets) return fail(DARB_E_INVALID, "NULL buffer");
    if (ldw < p->N) return fail(DARB_E_INVALID, "ldw < N");
    return launched(launch_decode(*p, wdtype, values, offsets, W_out, ldw,
                                  static_cast<hipStream_t>(stream)), "decode launch");
}

int darb_spmv(const darb_plan *p, int wdtype, const void *values, const uint8_t *offsets,
              int xdtype, const void *x, float *y, void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    rc = check_product_dtypes(wdtype, xdtype);
    if (rc) return rc;
    if (!values || !offsets || !x || !y) return fail(DARB_E_INVALID, "NULL buffer");
    return launched(launch_spmv(*p, wdtype, values, offsets, nullptr, xdtype, x, y,
                                static_cast<hipStream_t>(stream)), "spmv launch");
}

static int check_batch(int64_t B, int64_t ldx, int64_t ldy) {
    if (B < 1 || B >= (int64_t(1) << 31)) return fail(DARB_E_INVALID, "B must be in [1, 2^31)");
    if (ldx < B) return fail(DARB_E_INVALID, "ldx < B");
    if (ldy < B) return fail(DARB_E_INVALID, "ldy < B");
    return DARB_OK;
}

int darb_spmm(const darb_plan *p, int wdtype, const void *values, const uint8_t *offsets,
              int xdtype, int64_t B, const void *X, int64_t ldx, float *Y, int64_t ldy,
              void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    rc = check_product_dtypes(wdtype, xdtype);
    if (rc) return rc;
    if (!values || !offsets || !X || !Y) return fail(DARB_E_INVALID, "NULL buffer");
    rc = check_batch(B, ldx, ldy);
    if (rc) return rc;
    return launched(launch_spmm(*p, wdtype, values, offsets, nullptr, xdtype, B, X, ldx, Y, ldy,
                                static_cast<hipStream_t>(stream)), "spmm launch");
}

// The packed words: required (and 4-byte aligned) unless the plan has none.
static int check_packed(const darb_plan *p, const uint32_t *packed) {
    if (!packed && p->packed_words > 0) return fail(DARB_E_INVALID, "packed is NULL");
    if (reinterpret_cast<uintptr_t>(packed) & 3)
        return fail(DARB_E_INVALID, "packed must be 4-byte aligned");
    return DARB_OK;
}

int darb_pack_offsets(const darb_plan *p, const uint8_t *offsets, uint32_t *packed,
                      void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    if (!offsets) return fail(DARB_E_INVALID, "NULL buffer");
    rc = check_packed(p, packed);
    if (rc) return rc;
    return launched(launch_pack_offsets(*p, offsets, packed, static_cast<hipStream_t>(stream)),
                    "pack launch");
}

int darb_unpack_offsets(const darb_plan *p, const uint32_t *packed, uint8_t *offsets,
                        void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    if (!offsets) return fail(DARB_E_INVALID, "NULL buffer");
    rc = check_packed(p, packed);
    if (rc) return rc;
    return launched(launch_unpack_offsets(*p, packed, offsets, static_cast<hipStream_t>(stream)),
                    "unpack launch");
}

int darb_spmv_packed(const darb_plan *p, int wdtype, const void *values, const uint32_t *packed,
                     int xdtype, const void *x, float *y, void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    rc = check_product_dtypes(wdtype, xdtype);
    if (rc) return rc;
    if (!values || !x || !y) return fail(DARB_E_INVALID, "NULL buffer");
    rc = check_packed(p, packed);
    if (rc) return rc;
    return launched(launch_spmv(*p, wdtype, values, nullptr, packed, xdtype, x, y,
                                static_cast<hipStream_t>(stream)), "spmv (packed) launch");
}

int darb_spmm_packed(const darb_plan *p, int wdtype, const void *values, const uint32_t *packed,
                     int xdtype, int64_t B, const void *X, int64_t ldx, float *Y, int64_t ldy,
                     void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    rc = check_product_dtypes(wdtype, xdtype);
    if (rc) return rc;
    if (!values || !X || !Y) return fail(DARB_E_INVALID, "NULL buffer");
    rc = check_packed(p, packed);
    if (rc) return rc;
    rc = check_batch(B, ldx, ldy);
    if (rc) return rc;
    return launched(launch_spmm(*p, wdtype, values, nullptr, packed, xdtype, B, X, ldx, Y, ldy,
                                static_cast<hipStream_t>(stream)), "spmm (packed) launch");
}

int darb_quantize_i8(const darb_plan *p, int wdtype, const void *values, int8_t *codes,
                     float *scales, void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    if (!valid_dtype(wdtype)) return fail(DARB_E_DTYPE, "unknown weight dtype");
    if (!values || !codes || !scales) return fail(DARB_E_INVALID, "NULL buffer");
    return launched(launch_quantize_i8(*p, wdtype, values, codes, scales,
                                       static_cast<hipStream_t>(stream)), "quantize launch");
}

// INT8 products: the offsets come from exactly one of `offsets` (bytes) and
// `packed`; with offsets NULL, packed follows the packed products' rules.
static int check_i8_product(const darb_plan *p, const int8_t *codes, const float *scales,
                            const uint8_t *offsets, const uint32_t *packed, int xdtype) {
    if (!valid_dtype(xdtype)) return fail(DARB_E_DTYPE, "unknown activation dtype");
    if (!codes || !scales) return fail(DARB_E_INVALID, "NULL buffer");
    if (offsets && packed) return fail(DARB_E_INVALID, "pass offsets or packed, not both");
    return offsets ? DARB_OK : check_packed(p, packed);
}

int darb_spmv_i8(const darb_plan *p, const int8_t *codes, const float *scales,
                 const uint8_t *offsets, const uint32_t *packed, int xdtype, const void *x,
                 float *y, void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    rc = check_i8_product(p, codes, scales, offsets, packed, xdtype);
    if (rc) return rc;
    if (!x || !y) return fail(DARB_E_INVALID, "NULL buffer");
    return launched(launch_spmv_i8(*p, codes, scales, offsets, packed, xdtype, x, y,
                                   static_cast<hipStream_t>(stream)), "spmv (int8) launch");
}

int darb_spmm_i8(const darb_plan *p, const int8_t *codes, const float *scales,
                 const uint8_t *offsets, const uint32_t *packed, int xdtype, int64_t B,
                 const void *X, int64_t ldx, float *Y, int64_t ldy, void *stream) {
    clear_error();
    int rc = check_uploaded(p);
    if (rc) return rc;
    rc = check_i8_product(p, codes, scales, offsets, packed, xdtype);
    if (rc) return rc;
    if (!X || !Y) return fail(DARB_E_INVALID, "NULL buffer");
    rc = check_batch(B, ldx, ldy);
    if (rc) return rc;
    return launched(launch_spmm_i8(*p, codes, scales, offsets, packed, xdtype, B, X, ldx, Y, ldy,
                                   static_cast<hipStream_t>(stream)), "spmm (int8) launch");
}

int darb_prune_workspace(int64_t M, int64_t N, int wdtype, int64_t *bytes) {
    clear_error();
    if (!bytes) return fail(DARB_E_INVALID, "bytes is NULL");
    if (M < 1 || M >= (int64_t(1) << 31) || N < 1 || N >= (int64_t(1) << 31))
        return fail(DARB_E_INVALID, "M and N must be in [1, 2^31)");
    if (!valid_dtype(wdtype)) return fail(DARB_E_DTYPE, "unknown weight dtype");
    *bytes = prune_workspace_bytes(M, N, wdtype);
    return DARB_OK;
}

int darb_prune_counts(int64_t M, int64_t N, int wdtype, const void *W, int64_t ldw, int64_t k,
                      int64_t *counts, void *workspace, int64_t workspace_bytes, void *stream) {
    clear_error();
    if (M < 1 || M >= (int64_t(1) << 31) || N < 1 || N >= (int64_t(1) << 31))
        return fail(DARB_E_INVALID, "M and N must be in [1, 2^31)");
    if (!valid_dtype(wdtype)) return fail(DARB_E_DTYPE, "unknown weight dtype");
    if (!W || !counts || !workspace) return fail(DARB_E_INVALID, "NULL buffer");
    if (ldw < N) return fail(DARB_E_INVALID, "ldw < N");
    if (k < 0 || k > M * N) return fail(DARB_E_INVALID, "k must be in [0, M*N]");
    if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0)
        return fail(DARB_E_INVALID, "workspace must be 256-byte aligned");
    if ((reinterpret_cast<uintptr_t>(counts) & 7) != 0)
        return fail(DARB_E_INVALID, "counts must be 8-byte aligned");
    const int64_t need = prune_workspace_bytes(M, N, wdtype);
    if (workspace_bytes < need)
        return fail(DARB_E_WORKSPACE, "pruning workspace needs " + std::to_string(need) + " bytes");
    return launched(launch_prune_counts(M, N, wdtype, W, ldw, k, counts, workspace,
                                        static_cast<hipStream_t>(stream)), "prune launch");
}

int darb_prune_counts_noalloc(int64_t M, int64_t N, int wdtype, const void *W, int64_t ldw,
                              int64_t k, int64_t *counts, void *stream) {
    clear_error();
    if (M < 1 || M >= (int64_t(1) << 31) || N < 1 || N >= (int64_t(1) << 31))
        return fail(DARB_E_INVALID, "M and N must be in [1, 2^31)");
    if (!valid_dtype(wdtype)) return fail(DARB_E_DTYPE, "unknown weight dtype");
    if (!W || !counts) return fail(DARB_E_INVALID, "NULL buffer");
    if (ldw < N) return fail(DARB_E_INVALID, "ldw < N");
    if (k < 0 || k > M * N) return fail(DARB_E_INVALID, "k must be in [0, M*N]");
    if ((reinterpret_cast<uintptr_t>(counts) & 7) != 0)
        return fail(DARB_E_INVALID, "counts must be 8-byte aligned");
    const int64_t max_rows = prune_static_max_rows();
    if (M > max_rows)
        return fail(DARB_E_INVALID, "M = " + std::to_string(M) + " exceeds the fixed pruning "
                                    "scratch (at most " + std::to_string(max_rows) +
                                    " rows); use darb_prune_counts with a workspace");
    const hipError_t e = launch_prune_counts_static(M, N, wdtype, W, ldw, k, counts,
                                                    static_cast<hipStream_t>(stream));
    return launched(e, "prune launch (fixed scratch)");
}

// Workspace of the LSTM layer, in floats: U [4H x T*batch] and G [4H x batch].
static int64_t lstm_workspace_floats(int64_t H, int64_t T, int64_t batch) {
    return 4 * H * T * batch + 4 * H * batch;
}

static int lstm_check(const darb_plan *wih, const void *wih_values, const uint8_t *wih_offsets,
                      const darb_plan *whh, const void *whh_values, const uint8_t *whh_offsets,
                      int wdtype, int64_t H, int64_t T, int64_t batch, const float *x_seq,
                      float *h_seq, float *h, float *c, float *workspace,
                      int64_t workspace_floats) {
    int rc = check_uploaded(wih);
    if (rc) return rc;
    rc = check_uploaded(whh);
    if (rc) return rc;
    if (!valid_dtype(wdtype)) return fail(DARB_E_DTYPE, "unknown weight dtype");
    if (!wih_values || !wih_offsets || !whh_values || !whh_offsets || !x_seq || !h_seq || !h ||
        !c || !workspace)
        return fail(DARB_E_INVALID, "NULL buffer");
    if (H < 1 || T < 1 || batch < 1) return fail(DARB_E_INVALID, "H, T, batch must be >= 1");
    if (whh->M != 4 * H || whh->N != H) return fail(DARB_E_INVALID, "W_hh must be [4H x H]");
    if (wih->M != 4 * H) return fail(DARB_E_INVALID, "W_ih must have 4H rows");
    if (T * batch >= (int64_t(1) << 31)) return fail(DARB_E_INVALID, "T * batch too large");
    if ((reinterpret_cast<uintptr_t>(workspace) & 15) != 0)
        return fail(DARB_E_INVALID, "workspace must be 16-byte aligned");
    const int64_t need = lstm_workspace_floats(H, T, batch);
    if (workspace_floats < need)
        return fail(DARB_E_WORKSPACE, "lstm workspace needs " + std::to_string(need) + " floats");
    return DARB_OK;
}

// The time steps.  When every gate row of the recurrent matrix fits the fused
// step kernel, one launch per step computes the product and the cell of every
// hidden unit, reading h from one buffer and writing the other (h and, as the
// second buffer, the first H x batch floats of G); otherwise two launches per
// step: the recurrent product into G, then the cell.
static int lstm_steps(const darb_plan *whh, const void *whh_values, const uint8_t *whh_offsets,
                      int wdtype, int64_t H, int64_t T, int64_t batch, const float *U, float *G,
                      float *h_seq, float *h, float *c, hipStream_t s) {
    const int64_t TB = T * batch;
    if (lstm_step_fusable(*whh, batch, h, G)) {
        float *hb[2] = {h, G};
        for (int64_t t = 0; t < T; ++t) {
            int rc = launched(launch_lstm_step(*whh, wdtype, whh_values, whh_offsets, H, batch,
                                               hb[t & 1], U + t * batch, TB, c, hb[(t + 1) & 1],
                                               h_seq + t * batch, TB, s), "lstm step");
            if (rc) return rc;
        }
        if (T & 1) {            // the final state ended in the second buffer
            hipError_t e = hipMemcpyAsync(h, G, size_t(H * batch) * sizeof(float),
                                          hipMemcpyDeviceToDevice, s);
            if (e != hipSuccess)
                return fail(DARB_E_HIP, std::string("lstm state copy: ") + hipGetErrorString(e));
        }
        return DARB_OK;
    }
    for (int64_t t = 0; t < T; ++t) {
        int rc = launched(launch_spmm(*whh, wdtype, whh_values, whh_offsets, nullptr, DARB_F32,
                                      batch, h, batch, G, batch, s), "lstm recurrent product");
        if (rc) return rc;
        rc = launched(launch_lstm_cell(H, batch, G, U + t * batch, TB, h, c, h_seq + t * batch, TB,
                                       s), "lstm cell");
        if (rc) return rc;
    }
    return DARB_OK;
}

int darb_lstm_workspace(int64_t H, int64_t T, int64_t batch, int64_t *floats) {
    clear_error();
    if (!floats) return fail(DARB_E_INVALID, "floats is NULL");
    if (H < 1 || T < 1 || batch < 1) return fail(DARB_E_INVALID, "H, T, batch must be >= 1");
    *floats = lstm_workspace_floats(H, T, batch);
    return DARB_OK;
}

int darb_lstm_layer(const darb_plan *wih, const void *wih_values, const uint8_t *wih_offsets,
                    const darb_plan *whh, const void *whh_values, const uint8_t *whh_offsets,
                    int wdtype, int64_t H, int64_t T, int64_t batch, const float *x_seq,
                    float *h_seq, float *h, float *c, float *workspace,
                    int64_t workspace_floats, void *stream) {
    clear_error();
    int rc = lstm_check(wih, wih_values, wih_offsets, whh, whh_values, whh_offsets, wdtype, H, T,
                        batch, x_seq, h_seq, h, c, workspace, workspace_floats);
    if (rc) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t TB = T * batch;
    float *U = workspace;              // [4H x T*batch]: input products of every step
    float *G = workspace + 4 * H * TB; // [4H x batch]: recurrent product of one step
    rc = launched(launch_spmm(*wih, wdtype, wih_values, wih_offsets, nullptr, DARB_F32, TB, x_seq,
                              TB, U, TB, s), "lstm input product");
    if (rc) return rc;
    return lstm_steps(whh, whh_values, whh_offsets, wdtype, H, T, batch, U, G, h_seq, h, c, s);
}

int darb_stream_read(const void *buf, int64_t bytes, float *sink, void *stream) {
    clear_error();
    if (!buf || !sink || bytes <= 0 || (bytes & 15) || (reinterpret_cast<uintptr_t>(buf) & 15))
        return fail(DARB_E_INVALID, "buf/sink NULL or bytes/alignment not a multiple of 16");
    return launched(launch_stream_read(buf, bytes, sink, static_cast<hipStream_t>(stream)),
                    "stream read launch");
}

int darb_stream_read_shape(const void *buf, int64_t bytes, int threads, int vectors, float *sink,
                           void *stream) {
    clear_error();
    if (!buf || !sink || bytes <= 0 || (bytes & 15) || (reinterpret_cast<uintptr_t>(buf) & 15))
        return fail(DARB_E_INVALID, "buf/sink NULL or bytes/alignment not a multiple of 16");
    const hipError_t e = launch_stream_read_shape(buf, bytes, threads, vectors, sink,
                                                  static_cast<hipStream_t>(stream));
    if (e == hipErrorInvalidValue) return fail(DARB_E_INVALID, "no stream read of that shape");
    return launched(e, "stream read launch");
}

int darb_stream_copy(void *dst, const void *src, int64_t bytes, void *stream) {
    clear_error();
    if (!dst || !src || bytes <= 0 || (bytes & 15) || (reinterpret_cast<uintptr_t>(dst) & 15) ||
        (reinterpret_cast<uintptr_t>(src) & 15))
        return fail(DARB_E_INVALID, "dst/src NULL or bytes/alignment not a multiple of 16");
    return launched(launch_stream_copy(dst, src, bytes, static_cast<hipStream_t>(stream)),
                    "stream copy launch");
}

}  // extern "C"
