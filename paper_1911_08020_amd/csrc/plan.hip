// The plan built on the device from per-row kept counts (section 3.2): each row's
// block size from its density, the rows grouped by block size (ascending; original
// order inside a group) and each row's first slot -- the same plan darb_plan_create_counts
// builds on the host, written straight into the plan workspace.
//
// Rounding in integers.  With d = count / N, f = the largest power of two with
// f * count <= N (the largest with f * d <= 1): d is itself a power-of-two fraction when
// f * count == N, and then both directions give b = f; otherwise rounding the density
// up gives b = f and rounding it down b = 2f.  Floor mode always rounds up; paper mode
// rounds up when d >= D, i.e. count * M >= kept (D = kept / (M N)).  A row with count 0
// gets b_max; b is clamped to [b_min, b_max].  These are the host rule's results: the
// host compares fp64 quotients, and two distinct quotients of this size never round
// to the same double.
//
// Three launches: per-row block size and per-workgroup group counts; one workgroup scans
// those counts into group starts and each workgroup's first position per group (and
// writes the group summary the host reads back); each row then takes its place --
// workgroup start plus its rank among the workgroup's rows of the same group, counted
// with ballots -- which gives the storage order, the first slot and the per-row table.
#include "darb_internal.h"

namespace darb {
namespace {

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / kWave;
constexpr int kGroups = kMaxBins;               // log2 b = 0 .. 7

__device__ __forceinline__ int row_log2b_counts(int64_t c, int64_t N, int64_t M, int64_t kept,
                                                int mode, int lmin, int lmax) {
    if (c <= 0) return lmax;
    if (c > N) c = N;
    int l = 0;                                  // largest l with (c << l) <= N
    while (l < 62 && (c << (l + 1)) <= N) ++l;
    const bool exact = (c << l) == N;
    const bool up = (mode == DARB_ROUND_FLOOR) || (c * M >= kept);
    if (!up && !exact) ++l;
    return l < lmin ? lmin : (l > lmax ? lmax : l);
}

// Rank of this lane among the wave's active lanes below it with the same key, and
// the wave's count per key (every lane of the wave gets the same counts).
__device__ __forceinline__ int wave_rank(int key, bool active, int (&count)[kGroups]) {
    const uint64_t below = (uint64_t(1) << (threadIdx.x & (kWave - 1))) - 1;
    int rank = 0;
#pragma unroll
    for (int v = 0; v < kGroups; ++v) {
        const uint64_t m = __ballot(active && key == v);
        count[v] = __popcll(m);
        if (key == v) rank = __popcll(m & below);
    }
    return rank;
}

// Block sizes (into rowinfo's low byte) and each workgroup's row count per group.
__global__ __launch_bounds__(kPlanThreads) void plan_sizes_kernel(
    int64_t M, int64_t N, const int64_t *__restrict__ counts, int64_t kept, int mode, int lmin,
    int lmax, int64_t *__restrict__ rowinfo, int32_t *__restrict__ wg_counts) {
    __shared__ int part[kPlanWaves][kGroups];
    const int64_t r = int64_t(blockIdx.x) * kPlanThreads + threadIdx.x;
    const bool active = r < M;
    int l = 0;
    if (active) {
        l = row_log2b_counts(counts[r], N, M, kept, mode, lmin, lmax);
        rowinfo[r] = l;
    }
    int cnt[kGroups];
    wave_rank(l, active, cnt);
    const int wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0)
        for (int v = 0; v < kGroups; ++v) part[wave][v] = cnt[v];
    __syncthreads();
    if (threadIdx.x < kGroups) {
        int s = 0;
        for (int w = 0; w < kPlanWaves; ++w) s += part[w][threadIdx.x];
        wg_counts[int64_t(blockIdx.x) * kGroups + threadIdx.x] = s;
    }
}

// One workgroup: group sizes and starts, and each workgroup's first position in each
// group (overwriting wg_counts).  summary: rows, first_row, first_elem, first_word,
// 8 int64 each.
__global__ __launch_bounds__(kPlanThreads) void plan_scan_kernel(
    int64_t N, int64_t nwg, int32_t *__restrict__ wg_counts, int64_t *__restrict__ summary) {
    __shared__ int64_t total[kGroups];
    __shared__ int64_t start[kGroups];
    const int v = threadIdx.x / kWave;                   // one wave per group
    const int lane = threadIdx.x & (kWave - 1);
    if (v < kGroups) {
        // rows of group v, summed in chunks of 64 workgroups
        int64_t s = 0;
        for (int64_t b = lane; b < nwg; b += kWave) s += wg_counts[b * kGroups + v];
        for (int m = kWave / 2; m >= 1; m >>= 1) s += __shfl_xor(s, m, kWave);
        if (lane == 0) total[v] = s;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t row = 0, elem = 0, word = 0;
        for (int g = 0; g < kGroups; ++g) {
            const int64_t nblk = (N + (int64_t(1) << g) - 1) >> g;
            start[g] = row;
            summary[g] = total[g];
            summary[kGroups + g] = row;
            summary[2 * kGroups + g] = elem;
            summary[3 * kGroups + g] = word;
            row += total[g];
            elem += total[g] * nblk;
            word += (total[g] * nblk + 31) / 32 * g;
        }
    }
    __syncthreads();
    if (v < kGroups) {
        // exclusive scan of group v's per-workgroup counts, 64 workgroups at a time
        int64_t base = start[v];
        for (int64_t b0 = 0; b0 < nwg; b0 += kWave) {
            const int64_t b = b0 + lane;
            const int64_t c = b < nwg ? wg_counts[b * kGroups + v] : 0;
            int64_t incl = c;
            for (int m = 1; m < kWave; m <<= 1) {
                const int64_t t = __shfl_up(incl, m, kWave);
                if (lane >= m) incl += t;
            }
            if (b < nwg) wg_counts[b * kGroups + v] = int32_t(base + incl - c);
            base += __shfl(incl, kWave - 1, kWave);
        }
    }
}

// Each row's storage position: its workgroup's first position in its group plus its
// rank among the workgroup's earlier rows of that group.
__global__ __launch_bounds__(kPlanThreads) void plan_place_kernel(
    int64_t M, int64_t N, const int32_t *__restrict__ wg_start,
    const int64_t *__restrict__ summary, int64_t *__restrict__ rowinfo,
    int32_t *__restrict__ perm) {
    __shared__ int part[kPlanWaves][kGroups];
    const int64_t r = int64_t(blockIdx.x) * kPlanThreads + threadIdx.x;
    const bool active = r < M;
    const int l = active ? int(rowinfo[r] & 0xFF) : 0;
    int cnt[kGroups];
    const int rank = wave_rank(l, active, cnt);
    const int wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0)
        for (int v = 0; v < kGroups; ++v) part[wave][v] = cnt[v];
    __syncthreads();
    if (!active) return;
    int before = 0;                                      // earlier waves' rows of group l
    for (int w = 0; w < wave; ++w) before += part[w][l];
    const int64_t pos = int64_t(wg_start[int64_t(blockIdx.x) * kGroups + l]) + before + rank;
    const int64_t nblk = (N + (int64_t(1) << l) - 1) >> l;
    const int64_t slot = summary[2 * kGroups + l] + (pos - summary[kGroups + l]) * nblk;
    perm[pos] = int32_t(r);
    rowinfo[r] = (slot << 8) | l;
}

}  // namespace

int64_t plan_device_scratch_bytes(int64_t M) {
    const int64_t nwg = (M + kPlanThreads - 1) / kPlanThreads;
    return 4 * kGroups * int64_t(sizeof(int64_t)) + nwg * kGroups * int64_t(sizeof(int32_t));
}

hipError_t launch_plan_device(int64_t M, int64_t N, const int64_t *counts, int64_t kept, int mode,
                              int lmin, int lmax, int32_t *perm, int64_t *rowinfo, void *scratch,
                              hipStream_t s) {
    const int64_t nwg = (M + kPlanThreads - 1) / kPlanThreads;
    if (nwg > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    int64_t *summary = static_cast<int64_t *>(scratch);
    int32_t *wg_counts = reinterpret_cast<int32_t *>(summary + 4 * kGroups);
    hipLaunchKernelGGL(plan_sizes_kernel, dim3(unsigned(nwg)), dim3(kPlanThreads), 0, s, M, N,
                       counts, kept, mode, lmin, lmax, rowinfo, wg_counts);
    hipLaunchKernelGGL(plan_scan_kernel, dim3(1), dim3(kPlanThreads), 0, s, N, nwg, wg_counts,
                       summary);
    hipLaunchKernelGGL(plan_place_kernel, dim3(unsigned(nwg)), dim3(kPlanThreads), 0, s, M, N,
                       wg_counts, summary, rowinfo, perm);
    return hipGetLastError();
}

}  // namespace darb
