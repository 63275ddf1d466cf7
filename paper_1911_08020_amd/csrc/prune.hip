// Irregular magnitude pruning on the device: DARB's first step (section 3.2)
// needs only each row's kept count under a global top-K magnitude mask
// (irregular pruning keeps the K largest-magnitude weights, section 2).
//
// Magnitude is the key the block-max selection uses: the stored bits with the
// sign cleared, compared as unsigned integers (31 bits for fp32, 15 for fp16);
// among equal keys the lower flat index r*N + c is kept first.
//
// The K-th largest key t is found by a most-significant-digit radix select:
// digits of 11, 10 and 10 bits (fp32) or 8 and 7 bits (fp16).  A histogram pass
// counts the current digit of the keys that match the digits chosen so far (one
// LDS histogram per workgroup, four interleaved copies so lanes with equal digits
// rarely hit the same address; each workgroup then adds its non-zero bins into the
// global totals), and a one-workgroup kernel picks the digit where the count from
// the top reaches the remaining K.  Finally, per row, the keys > t are counted and
// the keys == t taken in flat order, which for row counts means rows in ascending
// order.
//
// Only the first pass streams all of W.  The second one (split) counts, per row,
// the keys whose first digit is above the chosen one and copies the keys whose
// first digit equals it -- the candidates, typically about 1 % of W -- with their
// rows into the workspace; the remaining digits and the final counts then read the
// candidates only.  Each workgroup gathers its candidates in LDS and reserves room
// for them with one atomic; if a workgroup's LDS or the workspace's candidate
// room overflows, every later pass streams W instead (the result is the same).
// Below 64 MiB of W the split pass is skipped: there a pass over W costs less than
// the extra launches.
// All state stays on the device; nothing returns to the host between passes.
#include "darb_internal.h"

namespace darb {
namespace {

constexpr int kHistThreads = 1024;
constexpr int kHistWaves = kHistThreads / kWave;
constexpr int kMaxDigitBits = 11;
constexpr int kCopies = 4;                          // LDS histogram copies per workgroup
constexpr int kMaxHistGroups = 512;

// Radix-select state, in the workspace.
struct PruneState {
    uint32_t prefix;        // the digits chosen so far; after the last pass, the key t
    uint32_t overflow;      // the candidates did not fit: later passes stream W
    int64_t k_rem;          // keys still to take at or below the prefix
    unsigned long long n_cand;   // candidates stored
    unsigned long long n_last;   // keys matching the prefix after the latest digit
};

constexpr int kSplitLds = 8192;                     // candidates a workgroup can hold
constexpr int kCandPerThread = 16;                  // candidate passes: keys per thread
constexpr int64_t kSplitMinBytes = int64_t(64) << 20;   // W size from which the split pays

template <typename Bits> struct PruneTraits;
template <> struct PruneTraits<uint32_t> {
    static constexpr int VEC = 4;
    static constexpr int KEY_BITS = 31;
    static constexpr uint32_t MAG = 0x7FFFFFFFu;
};
template <> struct PruneTraits<uint16_t> {
    static constexpr int VEC = 8;
    static constexpr int KEY_BITS = 15;
    static constexpr uint32_t MAG = 0x7FFFu;
};
constexpr int kUnroll = 4;

template <typename Bits, int VEC> struct alignas(16) PVec { Bits e[VEC]; };

// A wave's work unit is one segment of one row: kSegRounds rounds of kUnroll
// 16-byte loads per lane.
constexpr int kSegRounds = 4;
template <typename Bits> constexpr int64_t seg_width() {
    return int64_t(kSegRounds) * kUnroll * kWave * PruneTraits<Bits>::VEC;
}

// Stream the wave's segments: on_unit(r) when the wave starts a segment of row r
// (all lanes together), then round(keys, valid) for every round of the segment
// (all lanes together): the lane's kUnroll * VEC keys and a mask of those inside
// the segment.
template <typename Bits, bool ALIGNED, typename U, typename R>
__device__ __forceinline__ void for_each_round(const Bits *__restrict__ W, int64_t ldw,
                                               int64_t M, int64_t N, int64_t segs, U &&on_unit,
                                               R &&round) {
    using Tr = PruneTraits<Bits>;
    constexpr int VEC = Tr::VEC;
    constexpr int64_t STEP = int64_t(kUnroll) * kWave * VEC;
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int64_t gw = int64_t(blockIdx.x) * (blockDim.x / kWave) + threadIdx.x / kWave;
    const int64_t tw = int64_t(gridDim.x) * (blockDim.x / kWave);
    const int64_t units = M * segs;
    for (int64_t u = gw; u < units; u += tw) {          // wave-uniform
        const int64_t r = u / segs;
        const int64_t c_begin = (u - r * segs) * seg_width<Bits>();
        const int64_t c_end = c_begin + seg_width<Bits>() < N ? c_begin + seg_width<Bits>() : N;
        const Bits *row = W + r * ldw;
        on_unit(r);
        for (int64_t c0 = c_begin; c0 < c_end; c0 += STEP) {
            PVec<Bits, VEC> v[kUnroll];
            uint32_t valid[kUnroll];                  // bit e: element e is inside the segment
#pragma unroll
            for (int q = 0; q < kUnroll; ++q) {
                const int64_t c = c0 + int64_t(q) * kWave * VEC + int64_t(lane) * VEC;
                if (ALIGNED && c + VEC <= c_end) {
                    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                    const u32x4 t = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x4 *>(row + c));
                    v[q] = __builtin_bit_cast(PVec<Bits, VEC>, t);
                    valid[q] = (1u << VEC) - 1u;
                } else {
                    valid[q] = 0;
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const bool in = c + e < c_end;
                        v[q].e[e] = in ? row[c + e] : Bits(0);
                        valid[q] |= in ? (1u << e) : 0u;
                    }
                }
            }
            uint32_t keys[kUnroll * VEC];
            uint32_t mask = 0;
#pragma unroll
            for (int q = 0; q < kUnroll; ++q) {
#pragma unroll
                for (int e = 0; e < VEC; ++e) keys[q * VEC + e] = uint32_t(v[q].e[e]) & Tr::MAG;
                mask |= valid[q] << (q * VEC);
            }
            round(keys, mask);
        }
    }
}

// As for_each_round, with f(key) for every element inside the segment (per lane).
template <typename Bits, bool ALIGNED, typename U, typename F>
__device__ __forceinline__ void for_each_key(const Bits *__restrict__ W, int64_t ldw, int64_t M,
                                             int64_t N, int64_t segs, U &&on_unit, F &&f) {
    constexpr int K = kUnroll * PruneTraits<Bits>::VEC;
    for_each_round<Bits, ALIGNED>(W, ldw, M, N, segs, on_unit,
                                  [&](const uint32_t (&keys)[K], uint32_t mask) {
#pragma unroll
                                      for (int j = 0; j < K; ++j)
                                          if (mask & (1u << j)) f(keys[j]);
                                  });
}

// Histogram of digit (key >> shift) & (2^width - 1) over keys whose higher bits
// (key >> (shift + width)) equal state.prefix, added into `total` (zeroed before
// the pass): each workgroup adds its non-zero bins once.  The keys come from W
// (all of it) or, when `from_cand` and the candidates fit, from the candidates.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_hist_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t segs, int shift,
    int width, const PruneState *__restrict__ st, unsigned long long *__restrict__ total,
    const uint64_t *__restrict__ cand, int from_cand) {
    constexpr int kStride = (1 << kMaxDigitBits) + 1;   // copies land in different banks
    __shared__ uint32_t hist[kCopies * kStride];
    const int bins = 1 << width;
    for (int i = int(threadIdx.x); i < kCopies * kStride; i += kHistThreads) hist[i] = 0;
    __syncthreads();
    const uint32_t prefix = st->prefix;
    const int hi = shift + width;                       // <= key bits <= 31
    const uint32_t dmask = uint32_t(bins - 1);
    uint32_t *mine = hist + (int(threadIdx.x) & (kCopies - 1)) * kStride;
    auto add = [&](uint32_t key) {
        if ((key >> hi) == prefix) atomicAdd(&mine[(key >> shift) & dmask], 1u);
    };
    if (from_cand && !st->overflow) {                   // uniform
        // kCandPerThread candidates per thread: few workgroups, so few bins to flush
        const uint64_t n = st->n_cand;
        const uint64_t per_group = uint64_t(kCandPerThread) * kHistThreads;
        if (uint64_t(blockIdx.x) * per_group >= n && blockIdx.x > 0) return;   // uniform
        const uint64_t groups = (n + per_group - 1) / per_group;
        const uint64_t stride = (groups < gridDim.x ? groups : gridDim.x) * kHistThreads;
        for (uint64_t i = uint64_t(blockIdx.x) * kHistThreads + threadIdx.x; i < n; i += stride)
            add(uint32_t(cand[i]));
    } else {
        for_each_key<Bits, ALIGNED>(W, ldw, M, N, segs, [](int64_t) {}, add);
    }
    __syncthreads();
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) {
        uint32_t s = 0;
#pragma unroll
        for (int c = 0; c < kCopies; ++c) s += hist[c * kStride + b];
        if (s) atomicAdd(&total[b], (unsigned long long)s);
    }
}

// The split pass, after the first digit d (= state.prefix) is chosen: per row, the
// keys with first digit > d go to gt1; keys with first digit == d are stored as
// (row << 32 | key) candidates.  Runs in the same grid as the histogram passes.
// If any workgroup's candidates overflow its LDS or the workspace's room, the
// state's overflow flag sends the later passes back to W.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_split_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t segs, int shift,
    PruneState *__restrict__ st, unsigned long long *__restrict__ gt1,
    uint64_t *__restrict__ cand, uint64_t cap) {
    __shared__ uint64_t buf[kSplitLds];
    __shared__ uint32_t n_buf;
    __shared__ uint64_t base;
    if (threadIdx.x == 0) n_buf = 0;
    __syncthreads();
    const uint32_t d = st->prefix;
    const int lane = int(threadIdx.x) & (kWave - 1);
    int64_t cur = -1;
    uint32_t n_gt = 0;
    auto flush = [&]() {
        uint32_t g = n_gt;
#pragma unroll
        for (int m = kWave / 2; m >= 1; m >>= 1) g += __shfl_xor(g, m, kWave);
        if (lane == 0 && cur >= 0 && g) atomicAdd(&gt1[cur], (unsigned long long)g);
        n_gt = 0;
    };
    constexpr int K = kUnroll * PruneTraits<Bits>::VEC;
    for_each_round<Bits, ALIGNED>(
        W, ldw, M, N, segs,
        [&](int64_t r) {
            if (r != cur) {
                flush();
                cur = r;
            }
        },
        [&](const uint32_t (&keys)[K], uint32_t mask) {
            // branch-free over the round's keys: the count above d and a mask of the
            // candidates; then one wave scan and one LDS atomic place them all
            uint32_t cm = 0;
#pragma unroll
            for (int j = 0; j < K; ++j) {
                const uint32_t top = keys[j] >> shift;
                const bool in = (mask >> j) & 1u;
                n_gt += (in && top > d) ? 1u : 0u;
                cm |= (in && top == d) ? (1u << j) : 0u;
            }
            const uint32_t c = uint32_t(__popc(cm));
            uint32_t incl = c;
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                const uint32_t t = __shfl_up(incl, o, kWave);
                incl += lane >= o ? t : 0u;
            }
            const uint32_t total = __shfl(incl, kWave - 1, kWave);
            if (total) {                                // wave-uniform
                uint32_t at = 0;
                if (lane == 0) at = atomicAdd(&n_buf, total);
                at = __shfl(at, 0, kWave);
                uint32_t pos = at + incl - c;
                while (cm) {
                    const int j = __ffs(cm) - 1;
                    cm &= cm - 1u;
                    if (pos < kSplitLds) buf[pos] = (uint64_t(cur) << 32) | keys[j];
                    ++pos;
                }
            }
        });
    flush();
    __syncthreads();
    const uint32_t n = n_buf;
    if (threadIdx.x == 0) {
        base = 0;
        if (n > kSplitLds) {
            atomicExch(&st->overflow, 1u);
        } else if (n > 0) {
            base = atomicAdd(&st->n_cand, (unsigned long long)n);
            if (base + n > cap) atomicExch(&st->overflow, 1u);
        }
    }
    __syncthreads();
    if (n <= kSplitLds && base + n <= cap)
        for (uint32_t i = threadIdx.x; i < n; i += kHistThreads) cand[base + i] = buf[i];
}

// Block-wide inclusive scan of one value per thread (kHistThreads threads).
__device__ __forceinline__ uint64_t block_inclusive_scan(uint64_t v, uint64_t *wave_tot) {
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int wave = int(threadIdx.x) / kWave;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint64_t o = __shfl_up(v, d, kWave);
        if (lane >= d) v += o;
    }
    if (lane == kWave - 1) wave_tot[wave] = v;
    __syncthreads();
    uint64_t before = 0;
    for (int w = 0; w < wave; ++w) before += wave_tot[w];
    __syncthreads();
    return v + before;
}

// One workgroup: find the digit d where the count of matching keys with digit > d
// is < k_rem <= that count plus total[d]; then clear `total` for the next pass.
__global__ __launch_bounds__(kHistThreads) void prune_select_kernel(
    uint64_t *__restrict__ total, int width, PruneState *__restrict__ st) {
    __shared__ uint64_t tot[1 << kMaxDigitBits];
    __shared__ uint64_t wave_tot[kHistWaves];
    const int bins = 1 << width;
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) {
        tot[b] = total[b];
        total[b] = 0;
    }
    __syncthreads();
    const int64_t k_rem = st->k_rem;
    const uint32_t prefix = st->prefix;
    __syncthreads();                                    // every thread has read the state
    // thread t owns the digits bins-1-2t and bins-2-2t (descending order)
    const int d0 = bins - 1 - 2 * int(threadIdx.x), d1 = d0 - 1;
    const uint64_t a = d0 >= 0 ? tot[d0] : 0, b = d1 >= 0 ? tot[d1] : 0;
    const uint64_t incl = block_inclusive_scan(a + b, wave_tot);
    const uint64_t excl = incl - a - b;
    const uint64_t k = uint64_t(k_rem);
    if (excl < k && k <= incl) {                        // exactly one thread
        uint32_t d;
        uint64_t above;
        if (k <= excl + a) {
            d = uint32_t(d0);
            above = excl;
        } else {
            d = uint32_t(d1);
            above = excl + a;
        }
        st->prefix = (prefix << width) | d;
        st->k_rem = int64_t(k - above);
        st->n_last = d == uint32_t(d0) ? a : b;
    }
}

// Per-row counts of keys > t (into counts) and == t (into eq); t = state.prefix.
// From the candidates when they fit (plus the split pass's gt1), else from W.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_count_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t segs,
    const PruneState *__restrict__ st, unsigned long long *__restrict__ gt,
    unsigned long long *__restrict__ eq, const uint64_t *__restrict__ cand,
    const unsigned long long *__restrict__ gt1) {
    const uint32_t t = st->prefix;
    // when every key equal to t is taken (always, without ties), they count with the
    // keys above t and the finish scan has nothing to do
    unsigned long long *__restrict__ eqc =
        st->n_last == (unsigned long long)st->k_rem ? gt : eq;
    if (!st->overflow) {                                // uniform
        // one candidate per thread; a workgroup's candidates are stored together and
        // cover few rows, so a wave's 64 usually share one row: then one atomic each
        const uint64_t n = st->n_cand;
        const uint64_t stride = uint64_t(gridDim.x) * kHistThreads;
        const uint64_t first = uint64_t(blockIdx.x) * kHistThreads + threadIdx.x;
        const int lane = int(threadIdx.x) & (kWave - 1);
        for (uint64_t i = first; i < n; i += stride) {
            const uint64_t c = cand[i];
            const uint32_t key = uint32_t(c);
            const int32_t r = int32_t(c >> 32);
            uint32_t g = key > t ? 1u : 0u, e = key == t ? 1u : 0u;
            const int32_t r0 = __builtin_amdgcn_readfirstlane(r);
            if (__all(r == r0)) {                       // wave-uniform
#pragma unroll
                for (int m = kWave / 2; m >= 1; m >>= 1) {
                    g += __shfl_xor(g, m, kWave);
                    e += __shfl_xor(e, m, kWave);
                }
                if (lane == __ffsll((unsigned long long)__ballot(1)) - 1) {
                    if (g) atomicAdd(&gt[r0], (unsigned long long)g);
                    if (e) atomicAdd(&eqc[r0], (unsigned long long)e);
                }
            } else {
                if (g) atomicAdd(&gt[r], 1ull);
                if (e) atomicAdd(&eqc[r], 1ull);
            }
        }
        for (uint64_t r = first; r < uint64_t(M); r += stride)
            if (gt1[r]) atomicAdd(&gt[r], gt1[r]);
        return;
    }
    const int lane = int(threadIdx.x) & (kWave - 1);
    int64_t cur = -1;
    uint32_t n_gt = 0, n_eq = 0;
    auto flush = [&]() {
        uint32_t g = n_gt, e = n_eq;
#pragma unroll
        for (int d = kWave / 2; d >= 1; d >>= 1) {
            g += __shfl_xor(g, d, kWave);
            e += __shfl_xor(e, d, kWave);
        }
        if (lane == 0 && cur >= 0) {
            if (g) atomicAdd(&gt[cur], (unsigned long long)g);
            if (e) atomicAdd(&eqc[cur], (unsigned long long)e);
        }
        n_gt = n_eq = 0;
    };
    // a unit is one segment of one row: flush the previous row's counts when the
    // wave moves on (all lanes take part in the reduction)
    for_each_key<Bits, ALIGNED>(
        W, ldw, M, N, segs,
        [&](int64_t r) {
            if (r != cur) {
                flush();
                cur = r;
            }
        },
        [&](uint32_t key) {
            n_gt += key > t ? 1u : 0u;
            n_eq += key == t ? 1u : 0u;
        });
    flush();
}

// counts[r] (= keys > t) += the keys == t taken in ascending row order, need in total.
__global__ __launch_bounds__(kHistThreads) void prune_finish_kernel(
    int64_t M, const PruneState *__restrict__ st, int64_t *__restrict__ counts,
    const int64_t *__restrict__ eq) {
    __shared__ uint64_t wave_tot[kHistWaves];
    __shared__ int64_t tile_total;
    const int64_t need = st->k_rem;
    if (st->n_last == uint64_t(need)) return;           // all taken by the count pass
    int64_t carry = 0;                                   // keys == t in rows before the tile
    for (int64_t base = 0; base < M; base += kHistThreads) {
        const int64_t r = base + threadIdx.x;
        const int64_t e = r < M ? eq[r] : 0;
        const int64_t incl = int64_t(block_inclusive_scan(uint64_t(e), wave_tot));
        const int64_t before = carry + incl - e;
        if (r < M) {
            int64_t take = need - before;
            take = take < 0 ? 0 : (take > e ? e : take);
            counts[r] += take;
        }
        // the tile total, from the last thread's inclusive sum
        if (threadIdx.x == kHistThreads - 1) tile_total = incl;
        __syncthreads();
        carry += tile_total;
        __syncthreads();
    }
}

// Zero counts, eq, gt1 and the digit totals, and set the state to (prefix 0,
// k_rem = k, no candidates; overflow set when the split pass will not run).
__global__ __launch_bounds__(256) void prune_init_kernel(int64_t M, int64_t k, PruneState *st,
                                                         int64_t *counts, int64_t *eq,
                                                         int64_t *gt1, uint64_t *total,
                                                         int split) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i < M) {
        counts[i] = 0;
        eq[i] = 0;
        gt1[i] = 0;
    }
    if (i < (int64_t(1) << kMaxDigitBits)) total[i] = 0;
    if (i == 0 && st) {
        st->prefix = 0;
        st->overflow = split ? 0u : 1u;
        st->k_rem = k;
        st->n_cand = 0;
        st->n_last = 0;
    }
}

int64_t align256(int64_t v) { return (v + 255) / 256 * 256; }

template <typename Bits> int64_t segments(int64_t N) {
    return (N + seg_width<Bits>() - 1) / seg_width<Bits>();
}

template <typename Bits> int hist_groups(int64_t M, int64_t N) {
    // enough waves for every unit up to kMaxHistGroups workgroups, and few enough
    // elements per workgroup that its 32-bit LDS counters cannot overflow
    const int64_t units = M * segments<Bits>(N);
    int64_t g = (units + kHistWaves - 1) / kHistWaves;
    if (g > kMaxHistGroups) g = kMaxHistGroups;
    const int64_t per_group_limit = int64_t(1) << 31;
    while (g * per_group_limit < M * N) g *= 2;
    return int(g < 1 ? 1 : g);
}

// Room for candidates: 1/32 of W's elements (typical candidates are ~1 %), at
// least 64 Ki (or all of W when smaller), at most 2^28.
int64_t cand_capacity(int64_t M, int64_t N) {
    const int64_t all = M * N;
    int64_t c = (all + 31) / 32;
    const int64_t lo = all < (int64_t(1) << 16) ? all : (int64_t(1) << 16);
    if (c < lo) c = lo;
    if (c > (int64_t(1) << 28)) c = int64_t(1) << 28;
    return c;
}

// Workspace: the state, the digit totals, the per-row counts of keys equal to the
// threshold and of keys above the first digit, then the candidates.
struct PruneWorkspace {
    PruneState *st;
    uint64_t *total;        // [2^kMaxDigitBits]
    int64_t *eq;            // [M]
    int64_t *gt1;           // [M]
    uint64_t *cand;         // [cand_capacity]
};

struct PruneOffsets { int64_t total, eq, gt1, cand, bytes; };

PruneOffsets prune_offsets(int64_t M, int64_t N) {
    PruneOffsets o;
    o.total = align256(int64_t(sizeof(PruneState)));
    o.eq = o.total + align256((int64_t(1) << kMaxDigitBits) * 8);
    o.gt1 = o.eq + align256(M * int64_t(sizeof(int64_t)));
    o.cand = o.gt1 + align256(M * int64_t(sizeof(int64_t)));
    o.bytes = o.cand + align256(cand_capacity(M, N) * int64_t(sizeof(uint64_t)));
    return o;
}

PruneWorkspace prune_workspace(int64_t M, int64_t N, void *base) {
    const PruneOffsets o = prune_offsets(M, N);
    char *c = static_cast<char *>(base);
    PruneWorkspace w;
    w.st = reinterpret_cast<PruneState *>(c);
    w.total = reinterpret_cast<uint64_t *>(c + o.total);
    w.eq = reinterpret_cast<int64_t *>(c + o.eq);
    w.gt1 = reinterpret_cast<int64_t *>(c + o.gt1);
    w.cand = reinterpret_cast<uint64_t *>(c + o.cand);
    return w;
}

template <typename Bits>
hipError_t launch_prune_t(int64_t M, int64_t N, const void *Wv, int64_t ldw, int64_t k,
                          int64_t *counts, void *workspace, hipStream_t s) {
    using Tr = PruneTraits<Bits>;
    const Bits *W = static_cast<const Bits *>(Wv);
    const PruneWorkspace w = prune_workspace(M, N, workspace);
    PruneState *st = w.st;
    int64_t *eq = w.eq;
    auto *total_u = reinterpret_cast<unsigned long long *>(w.total);
    const int groups = hist_groups<Bits>(M, N);
    const int64_t init_n = M > (int64_t(1) << kMaxDigitBits) ? M : (int64_t(1) << kMaxDigitBits);
    const int64_t init_blocks = (init_n + 255) / 256;
    if (init_blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    // the split pass pays for its extra launches only on large matrices: below
    // kSplitMinBytes of W every pass streams W
    const int split = M * N * int64_t(sizeof(Bits)) >= kSplitMinBytes ? 1 : 0;
    hipLaunchKernelGGL(prune_init_kernel, dim3(unsigned(init_blocks)), dim3(256), 0, s, M, k, st,
                       counts, eq, w.gt1, w.total, split);
    if (k == 0) return hipGetLastError();               // nothing kept: counts stay 0

    const int64_t segs = segments<Bits>(N);
    const bool aligned = (reinterpret_cast<uintptr_t>(W) % 16 == 0) &&
                         ((ldw * int64_t(sizeof(Bits))) % 16 == 0);
    // digit widths from the most significant end
    const int widths32[3] = {11, 10, 10}, widths16[2] = {8, 7};
    const int *widths = Tr::KEY_BITS == 31 ? widths32 : widths16;
    const int passes = Tr::KEY_BITS == 31 ? 3 : 2;
    const uint64_t cap = uint64_t(cand_capacity(M, N));
    auto *gt1_u = reinterpret_cast<unsigned long long *>(w.gt1);
    int hi = Tr::KEY_BITS;
    for (int p = 0; p < passes; ++p) {
        const int width = widths[p];
        const int shift = hi - width;
        const int from_cand = p > 0;
        if (aligned)
            hipLaunchKernelGGL((prune_hist_kernel<Bits, true>), dim3(groups), dim3(kHistThreads),
                               0, s, W, ldw, M, N, segs, shift, width, st, total_u, w.cand,
                               from_cand);
        else
            hipLaunchKernelGGL((prune_hist_kernel<Bits, false>), dim3(groups), dim3(kHistThreads),
                               0, s, W, ldw, M, N, segs, shift, width, st, total_u, w.cand,
                               from_cand);
        hipLaunchKernelGGL(prune_select_kernel, dim3(1), dim3(kHistThreads), 0, s, w.total, width,
                           st);
        if (p == 0 && split) {                          // first digit chosen: split W once
            if (aligned)
                hipLaunchKernelGGL((prune_split_kernel<Bits, true>), dim3(groups),
                                   dim3(kHistThreads), 0, s, W, ldw, M, N, segs, shift, st,
                                   gt1_u, w.cand, cap);
            else
                hipLaunchKernelGGL((prune_split_kernel<Bits, false>), dim3(groups),
                                   dim3(kHistThreads), 0, s, W, ldw, M, N, segs, shift, st,
                                   gt1_u, w.cand, cap);
        }
        hi = shift;
    }
    auto *gt_u = reinterpret_cast<unsigned long long *>(counts);
    auto *eq_u = reinterpret_cast<unsigned long long *>(eq);
    if (aligned)
        hipLaunchKernelGGL((prune_count_kernel<Bits, true>), dim3(groups), dim3(kHistThreads), 0,
                           s, W, ldw, M, N, segs, st, gt_u, eq_u, w.cand, gt1_u);
    else
        hipLaunchKernelGGL((prune_count_kernel<Bits, false>), dim3(groups), dim3(kHistThreads), 0,
                           s, W, ldw, M, N, segs, st, gt_u, eq_u, w.cand, gt1_u);
    hipLaunchKernelGGL(prune_finish_kernel, dim3(1), dim3(kHistThreads), 0, s, M, st, counts, eq);
    return hipGetLastError();
}

}  // namespace

int64_t prune_workspace_bytes(int64_t M, int64_t N, int wdtype) {
    (void)wdtype;
    return prune_offsets(M, N).bytes;
}

hipError_t launch_prune_counts(int64_t M, int64_t N, int wdtype, const void *W, int64_t ldw,
                               int64_t k, int64_t *counts, void *workspace, hipStream_t s) {
    if (wdtype == DARB_F32) return launch_prune_t<uint32_t>(M, N, W, ldw, k, counts, workspace, s);
    return launch_prune_t<uint16_t>(M, N, W, ldw, k, counts, workspace, s);
}

}  // namespace darb
