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
// global totals), and the workgroup that finishes the pass last (a counter in the
// state tells it) picks the digit where the count from the top reaches the
// remaining K.  Finally, per row, the keys > t are counted and the keys == t taken
// in flat order, which for row counts means rows in ascending order (by the count
// pass's last workgroup).
//
// From 64 MiB of W one pass streams all of W.  A sample of W (about 1/32) first
// proposes a bracket of first digits that holds the K-th key's, with a margin of
// six binomial standard deviations.  The split pass then counts, per row, the keys
// whose first digit is above the bracket and copies the keys inside it -- the
// candidates, typically about 1 % of W -- with their rows into the workspace; it
// also takes the exact first-digit histogram, and its last workgroup picks the
// first digit and checks it against the bracket.  The remaining digits and the
// final counts read the candidates only.  Each workgroup gathers its candidates in
// LDS and reserves room for them with one atomic; if a workgroup's LDS or the
// workspace's candidate room overflows, or the first digit lies outside the
// bracket, every later pass streams W instead (the result is the same).  When the
// sample predicts more candidates than half the room, the exact first-digit
// histogram runs over W before the split, which then keeps that digit only.
// Below 64 MiB of W there is no sample and no split: every pass streams W, which
// there costs less than the extra launches.
// All state stays on the device; nothing returns to the host between passes.
#include <algorithm>

#include <mutex>

#include "darb_internal.h"

namespace darb {
namespace {

constexpr int kHistThreads = 1024;
constexpr int kHistWaves = kHistThreads / kWave;
constexpr int kMaxDigitBits = 11;
constexpr int kCopies = 4;                          // LDS histogram copies per workgroup
constexpr int kMaxHistGroups = 256;                 // one 1024-thread workgroup per CU

// Radix-select state, in the workspace.
struct PruneState {
    uint32_t prefix;        // the digits chosen so far; after the last pass, the key t
    uint32_t overflow;      // the candidates did not fit: later passes stream W
    int64_t k_rem;          // keys still to take at or below the prefix
    unsigned long long n_cand;   // candidates stored
    unsigned long long n_last;   // keys matching the prefix after the latest digit
    uint32_t done;          // workgroups finished in the running pass (0 between passes)
    uint32_t single;        // the split pass also takes the first digit's histogram
    uint32_t dlo, dhi;      // first digits the split pass keeps as candidates
};

constexpr int kSplitLds = 8192;                     // candidates a workgroup can hold
constexpr int64_t kSampleEvery = 32;                // the sample reads about 1/32 of W
constexpr int64_t kSampleDrift = 37;                // vectors added to the sample stride
constexpr int64_t kSampleChunk = 4;                 // vectors per lane in one sampled range
constexpr int kSampleGroups = 256;                  // workgroups of the sample pass
constexpr int kCandPerThread = 16;                  // candidate passes: keys per thread
constexpr int64_t kSplitMinBytes = int64_t(64) << 20;   // W size from which the split pays

template <typename Bits> struct PruneTraits;
template <> struct PruneTraits<uint32_t> {
    static constexpr int VEC = 4;
    static constexpr int UNROLL = 4;        // 16-byte loads per lane per round
    static constexpr int KEY_BITS = 31;
    static constexpr uint32_t MAG = 0x7FFFFFFFu;
};
template <> struct PruneTraits<uint16_t> {
    static constexpr int VEC = 8;
    static constexpr int UNROLL = 2;        // 16 keys per lane per round, as for fp32
    static constexpr int KEY_BITS = 15;
    static constexpr uint32_t MAG = 0x7FFFu;
};

template <typename Bits, int VEC> struct alignas(16) PVec { Bits e[VEC]; };

// Work is split evenly over the waves: W is taken as M rows padded to whole
// VEC-element vectors, flattened, and wave w streams elements [w * per_wave,
// (w + 1) * per_wave) of that (per_wave a multiple of kWave * VEC, so every piece
// starts on a vector boundary), in pieces of one row each.  A sample reads ranges
// of per_wave elements range_stride apart instead (range_stride = per_wave reads
// all of W).
template <typename Bits> constexpr int64_t round_width() {
    return int64_t(PruneTraits<Bits>::UNROLL) * kWave * PruneTraits<Bits>::VEC;
}
template <typename Bits> __host__ __device__ constexpr int64_t padded_n(int64_t N) {
    return (N + PruneTraits<Bits>::VEC - 1) / PruneTraits<Bits>::VEC * PruneTraits<Bits>::VEC;
}

// Stream the wave's pieces: on_unit(r) when the wave starts a piece of row r
// (all lanes together), then round(keys, valid) for every round of the piece
// (all lanes together): the lane's kUnroll * VEC keys and a mask of those inside
// the row.
template <typename Bits, bool ALIGNED, typename U, typename R>
__device__ __forceinline__ void for_each_round(const Bits *__restrict__ W, int64_t ldw,
                                               int64_t M, int64_t N, int64_t per_wave,
                                               int64_t range_stride, U &&on_unit, R &&round) {
    using Tr = PruneTraits<Bits>;
    constexpr int VEC = Tr::VEC;
    constexpr int kUnroll = Tr::UNROLL;
    constexpr int64_t STEP = round_width<Bits>();
    const int lane = int(threadIdx.x) & (kWave - 1);
    // the wave's index, made visibly wave-uniform so the loop state stays scalar
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
    const int64_t gw = int64_t(blockIdx.x) * (blockDim.x / kWave) + wave;
    const int64_t tw = int64_t(gridDim.x) * (blockDim.x / kWave);
    const int64_t Np = padded_n<Bits>(N);
    const int64_t total = M * Np;
    for (int64_t a = gw * range_stride; a < total; a += tw * range_stride) {   // wave-uniform
        const int64_t b = a + per_wave < total ? a + per_wave : total;
        int64_t r = a / Np;
        int64_t c = a - r * Np;
        for (int64_t at = a; at < b; ++r, c = 0) {
            const int64_t c_piece = c + (b - at) < Np ? c + (b - at) : Np;
            const int64_t c_end = c_piece < N ? c_piece : N;
            at += c_piece - c;
            const Bits *row = W + r * ldw;
            on_unit(r);
            for (int64_t c0 = c; c0 < c_end; c0 += STEP) {
                PVec<Bits, VEC> v[kUnroll];
                uint32_t valid[kUnroll];              // bit e: element e is inside the row
#pragma unroll
                for (int q = 0; q < kUnroll; ++q) {
                    const int64_t cc = c0 + int64_t(q) * kWave * VEC + int64_t(lane) * VEC;
                    // a vector wholly past the end costs nothing (and, unlike the
                    // element path, does not wait for the round's other loads)
                    if (cc >= c_end) {
                        v[q] = PVec<Bits, VEC>{};
                        valid[q] = 0;
                    } else if (ALIGNED && cc + VEC <= c_end) {
                        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                        const u32x4 t = __builtin_nontemporal_load(
                            reinterpret_cast<const u32x4 *>(row + cc));
                        v[q] = __builtin_bit_cast(PVec<Bits, VEC>, t);
                        valid[q] = (1u << VEC) - 1u;
                    } else {
                        valid[q] = 0;
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            const bool in = cc + e < c_end;
                            v[q].e[e] = in ? row[cc + e] : Bits(0);
                            valid[q] |= in ? (1u << e) : 0u;
                        }
                    }
                }
                uint32_t keys[kUnroll * VEC];
                uint32_t mask = 0;
#pragma unroll
                for (int q = 0; q < kUnroll; ++q) {
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        keys[q * VEC + e] = uint32_t(v[q].e[e]) & Tr::MAG;
                    mask |= valid[q] << (q * VEC);
                }
                round(keys, mask);
            }
        }
    }
}

// As for_each_round, with f(key) for every element inside the row (per lane).
template <typename Bits, bool ALIGNED, typename U, typename F>
__device__ __forceinline__ void for_each_key(const Bits *__restrict__ W, int64_t ldw, int64_t M,
                                             int64_t N, int64_t per_wave, int64_t range_stride,
                                             U &&on_unit, F &&f) {
    constexpr int K = PruneTraits<Bits>::UNROLL * PruneTraits<Bits>::VEC;
    for_each_round<Bits, ALIGNED>(W, ldw, M, N, per_wave, range_stride, on_unit,
                                  [&](const uint32_t (&keys)[K], uint32_t mask) {
#pragma unroll
                                      for (int j = 0; j < K; ++j)
                                          if (mask & (1u << j)) f(keys[j]);
                                  });
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

// Called by every thread of a workgroup after its global atomics: true in the
// one workgroup that finishes the pass last, which also clears the counter for
// the next pass.  Every value that crosses workgroups goes through device-wide
// read-modify-write atomics, which are coherent across the chip's L2 caches: each
// thread waits until its own atomics are acknowledged before the barrier, so they
// precede the workgroup's increment of the counter, and the last workgroup reads
// the totals with read-modify-write atomics too.  (An agent-scope fence would
// write back and invalidate the L2 in every wave of every workgroup.)
__device__ __forceinline__ bool last_workgroup(PruneState *st, uint32_t *flag) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t before = atomicAdd(&st->done, 1u);
        const bool last = before == gridDim.x - 1;
        if (last) atomicExch(&st->done, 0u);
        *flag = last ? 1u : 0u;
    }
    __syncthreads();
    return *flag != 0;
}

// What the workgroup that picks the first digit does with it besides.
enum SelectAfter { kJustSelect = 0, kSetBracket = 1, kCheckBracket = 2 };

// One workgroup, after a histogram pass: find the digit d where the count of
// matching keys with digit > d is < k_rem <= that count plus total[d], append it
// to the prefix, and clear `total` for the next pass.  For the first digit, also
// make d the split pass's bracket (kSetBracket), or, when the split pass took
// candidates from a sampled bracket, send the later passes back to W if d lies
// outside it (kCheckBracket).
__device__ __forceinline__ void select_digit(unsigned long long *__restrict__ total, int width,
                                             PruneState *__restrict__ st, uint64_t *tot,
                                             uint64_t *wave_tot, int after) {
    const int bins = 1 << width;
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) tot[b] = atomicExch(&total[b], 0ull);
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
        if (after == kSetBracket) {
            st->dlo = d;
            st->dhi = d;
        } else if (after == kCheckBracket && (d < st->dlo || d > st->dhi)) {
            atomicExch(&st->overflow, 1u);
        }
    }
}

// One workgroup, after the sample's first-digit histogram (n_s keys out of the
// matrix's total_keys, a fraction f): the split pass's bracket [dlo, dhi] of first
// digits that holds the k-th largest key's digit, up to six standard deviations
// of the sample count (a binomial) plus 8 keys: keys above dhi number at most
// f*k - margin in the sample, keys at or above dlo at least f*k + margin.  One pass
// over W then suffices (`single`) unless the bracket's predicted candidates exceed
// cand_limit.  Clears `total`.
__device__ __forceinline__ void select_bracket(unsigned long long *__restrict__ total, int width,
                                               PruneState *__restrict__ st, int64_t total_keys,
                                               uint64_t cand_limit, uint64_t *tot,
                                               uint64_t *wave_tot, uint32_t *lds_u32) {
    const int bins = 1 << width;
    uint32_t &s_dlo = lds_u32[0], &s_dhi = lds_u32[1];
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) tot[b] = atomicExch(&total[b], 0ull);
    if (threadIdx.x == 0) {
        s_dlo = 0;
        s_dhi = uint32_t(bins - 1);
    }
    __syncthreads();
    const double k = double(st->k_rem);
    // thread t owns the digits bins-1-2t and bins-2-2t (descending order)
    const int d0 = bins - 1 - 2 * int(threadIdx.x), d1 = d0 - 1;
    const uint64_t a = d0 >= 0 ? tot[d0] : 0, b = d1 >= 0 ? tot[d1] : 0;
    const uint64_t incl = block_inclusive_scan(a + b, wave_tot);
    const uint64_t excl = incl - a - b;
    uint64_t n_s = 0;
    for (int w = 0; w < kHistWaves; ++w) n_s += wave_tot[w];
    const double q = k / double(total_keys);
    const double ks = q * double(n_s);
    const double margin = 6.0 * sqrt(ks * (1.0 - q)) + 8.0;
    const double lo = ks - margin, hi = ks + margin;
    // digit d has `above` keys with a larger digit and `above + tot[d]` at or above
    // it, both non-increasing in d: dhi is the one digit with above <= lo <
    // above + tot[d] (or digit 0 with above <= lo), dlo the one with above < hi <=
    // above + tot[d] (or the top digit with tot >= hi); the defaults stand when no
    // digit qualifies.  One thread writes each (no contended atomics).
    auto ends = [&](int d, uint64_t above, uint64_t cnt) {
        if (d < 0) return;
        const double ab = double(above), at = double(above + cnt);
        if (ab <= lo && (d == 0 || at > lo)) s_dhi = uint32_t(d);
        if (at >= hi && (d == bins - 1 || ab < hi)) s_dlo = uint32_t(d);
    };
    ends(d0, excl, a);
    ends(d1, excl + a, b);
    __syncthreads();
    const uint32_t dlo = s_dlo, dhi = s_dhi;
    uint64_t in = 0;
    if (d0 >= 0 && uint32_t(d0) >= dlo && uint32_t(d0) <= dhi) in += a;
    if (d1 >= 0 && uint32_t(d1) >= dlo && uint32_t(d1) <= dhi) in += b;
    __syncthreads();                                    // wave_tot is reused
    const uint64_t in_all = block_inclusive_scan(in, wave_tot);
    if (threadIdx.x == kHistThreads - 1) {
        // predicted candidates: the bracket's sample keys scaled by 1/f
        const bool fits = n_s > 0 && double(in_all) * double(total_keys) <=
                                         double(cand_limit) * double(n_s);
        st->single = fits ? 1u : 0u;
        st->dlo = dlo;
        st->dhi = dhi;
    }
}

// What a histogram pass is for.
enum HistRole {
    kRoleDigit = 0,     // the next digit (W, or the candidates when they fit)
    kRoleSample = 1,    // the first digit over a sample of W: the split pass's bracket
    kRoleFirst = 2,     // the first digit over all of W, unless the bracket suffices
};

// Histogram of digit (key >> shift) & (2^width - 1) over keys whose higher bits
// (key >> (shift + width)) equal state.prefix, added into `total` (zero at the
// start): each workgroup adds its non-zero bins once, and the last workgroup to
// finish picks the digit (or, for the sample, the bracket).  The keys come from
// W (ranges of per_wave elements range_stride apart), or, when `from_cand` and
// the candidates fit, from the candidates.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_hist_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave,
    int64_t range_stride, int shift, int width, PruneState *__restrict__ st,
    unsigned long long *__restrict__ total, const uint64_t *__restrict__ cand, int from_cand,
    int role, uint64_t cand_limit) {
    constexpr int kStride = (1 << kMaxDigitBits) + 1;   // copies land in different banks
    __shared__ uint32_t hist[kCopies * kStride];
    __shared__ uint64_t tot[1 << kMaxDigitBits];
    __shared__ uint64_t wave_tot[kHistWaves];
    __shared__ uint32_t flag[3];                 // last-workgroup flag, bracket ends
    if (role == kRoleFirst && st->single) return;       // uniform: the split pass does it
    const int bins = 1 << width;
    const bool cands = from_cand && !st->overflow;     // uniform
    const uint64_t n = cands ? uint64_t(st->n_cand) : 0;
    // kCandPerThread candidates per thread: few workgroups, so few bins to flush
    const uint64_t per_group = uint64_t(kCandPerThread) * kHistThreads;
    const bool idle = cands && blockIdx.x > 0 && uint64_t(blockIdx.x) * per_group >= n;
    if (!idle) {                                        // uniform
        for (int i = int(threadIdx.x); i < kCopies * kStride; i += kHistThreads) hist[i] = 0;
        __syncthreads();
        const uint32_t prefix = st->prefix;
        const int hi = shift + width;                   // <= key bits <= 31
        const uint32_t dmask = uint32_t(bins - 1);
        uint32_t *mine = hist + (int(threadIdx.x) & (kCopies - 1)) * kStride;
        auto add = [&](uint32_t key) {
            if ((key >> hi) == prefix) atomicAdd(&mine[(key >> shift) & dmask], 1u);
        };
        if (cands) {
            const uint64_t groups = (n + per_group - 1) / per_group;
            const uint64_t stride = (groups < gridDim.x ? groups : gridDim.x) * kHistThreads;
            // all of a thread's loads issued before its LDS atomics
            for (uint64_t i0 = uint64_t(blockIdx.x) * kHistThreads + threadIdx.x; i0 < n;
                 i0 += stride * kCandPerThread) {
                uint32_t kk[kCandPerThread];
#pragma unroll
                for (int j = 0; j < kCandPerThread; ++j) {
                    const uint64_t i = i0 + uint64_t(j) * stride;
                    kk[j] = i < n ? uint32_t(cand[i]) : 0u;
                }
#pragma unroll
                for (int j = 0; j < kCandPerThread; ++j)
                    if (i0 + uint64_t(j) * stride < n) add(kk[j]);
            }
        } else {
            for_each_key<Bits, ALIGNED>(W, ldw, M, N, per_wave, range_stride, [](int64_t) {},
                                        add);
        }
        __syncthreads();
        for (int b = int(threadIdx.x); b < bins; b += kHistThreads) {
            uint32_t s = 0;
#pragma unroll
            for (int c = 0; c < kCopies; ++c) s += hist[c * kStride + b];
            if (s) atomicAdd(&total[b], (unsigned long long)s);
        }
    }
    if (!last_workgroup(st, &flag[0])) return;
    if (role == kRoleSample)
        select_bracket(total, width, st, M * N, cand_limit, tot, wave_tot, flag + 1);
    else
        select_digit(total, width, st, tot, wave_tot, role == kRoleFirst ? kSetBracket : kJustSelect);
}

// The split pass, once the bracket [dlo, dhi] of first digits is known: per row,
// the keys with first digit > dhi go to gt1; keys with first digit in the bracket
// are stored as (row << 32 | key) candidates.  Runs in the same grid as the
// histogram passes.  If any workgroup's candidates overflow its LDS or the
// workspace's room, the state's overflow flag sends the later passes back to W.
// With `single` (the bracket came from a sample) it also takes the first digit's
// histogram of all of W, and its last workgroup picks the digit and checks that
// it lies in the bracket (if not, the later passes go back to W as well).
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_split_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave, int shift,
    int width, PruneState *__restrict__ st, unsigned long long *__restrict__ gt1,
    uint64_t *__restrict__ cand, uint64_t cap, unsigned long long *__restrict__ total) {
    constexpr int kStride = (1 << kMaxDigitBits) + 1;
    __shared__ uint64_t buf[kSplitLds];
    __shared__ uint32_t hist[kCopies * kStride];
    __shared__ uint64_t tot[1 << kMaxDigitBits];
    __shared__ uint64_t wave_tot[kHistWaves];
    __shared__ uint32_t n_buf, flag;
    __shared__ uint64_t base;
    const bool single = st->single != 0;                // uniform
    const uint32_t dlo = st->dlo, dhi = st->dhi;
    const int bins = 1 << width;
    if (threadIdx.x == 0) n_buf = 0;
    if (single)
        for (int i = int(threadIdx.x); i < kCopies * kStride; i += kHistThreads) hist[i] = 0;
    __syncthreads();
    uint32_t *mine = hist + (int(threadIdx.x) & (kCopies - 1)) * kStride;
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
    constexpr int K = PruneTraits<Bits>::UNROLL * PruneTraits<Bits>::VEC;
    for_each_round<Bits, ALIGNED>(
        W, ldw, M, N, per_wave, per_wave,
        [&](int64_t r) {
            if (r != cur) {
                flush();
                cur = r;
            }
        },
        [&](const uint32_t (&keys)[K], uint32_t mask) {
            // branch-free over the round's keys: the count above the bracket and a
            // mask of the candidates; then one wave scan and one LDS atomic place
            // them all
            uint32_t cm = 0;
#pragma unroll
            for (int j = 0; j < K; ++j) {
                const uint32_t top = keys[j] >> shift;
                const bool in = (mask >> j) & 1u;
                n_gt += (in && top > dhi) ? 1u : 0u;
                cm |= (in && top >= dlo && top <= dhi) ? (1u << j) : 0u;
            }
            if (single) {                               // uniform
#pragma unroll
                for (int j = 0; j < K; ++j)
                    if ((mask >> j) & 1u) atomicAdd(&mine[keys[j] >> shift], 1u);
            }
            const uint32_t c = uint32_t(__popc(cm));
            uint32_t incl = c;
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                const uint32_t t = __shfl_up(incl, o, kWave);
                incl += lane >= o ? t : 0u;
            }
            const uint32_t total_c = __shfl(incl, kWave - 1, kWave);
            if (total_c) {                              // wave-uniform
                uint32_t at = 0;
                if (lane == 0) at = atomicAdd(&n_buf, total_c);
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
    if (!single) return;                                // uniform
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) {
        uint32_t s = 0;
#pragma unroll
        for (int c = 0; c < kCopies; ++c) s += hist[c * kStride + b];
        if (s) atomicAdd(&total[b], (unsigned long long)s);
    }
    if (last_workgroup(st, &flag)) select_digit(total, width, st, tot, wave_tot, kCheckBracket);
}

// counts[r] (= keys > t) += the keys == t taken in ascending row order, need in
// total; one workgroup.
__device__ __forceinline__ void take_ties(int64_t M, const PruneState *__restrict__ st,
                                          unsigned long long *__restrict__ counts,
                                          unsigned long long *__restrict__ eq,
                                          uint64_t *wave_tot, int64_t *tile_total) {
    const int64_t need = st->k_rem;
    int64_t carry = 0;                                   // keys == t in rows before the tile
    for (int64_t base = 0; base < M; base += kHistThreads) {
        const int64_t r = base + threadIdx.x;
        const int64_t e = r < M ? int64_t(atomicAdd(&eq[r], 0ull)) : 0;
        const int64_t incl = int64_t(block_inclusive_scan(uint64_t(e), wave_tot));
        const int64_t before = carry + incl - e;
        if (r < M) {
            int64_t take = need - before;
            take = take < 0 ? 0 : (take > e ? e : take);
            if (take) atomicAdd(&counts[r], (unsigned long long)take);
        }
        // the tile total, from the last thread's inclusive sum
        if (threadIdx.x == kHistThreads - 1) *tile_total = incl;
        __syncthreads();
        carry += *tile_total;
        __syncthreads();
    }
}

// Per-row counts of keys > t (into counts) and == t (into eq); t = state.prefix.
// From the candidates when they fit (plus the split pass's gt1), else from W.
// The last workgroup to finish then adds the keys == t that are kept.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_count_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave,
    PruneState *__restrict__ st, unsigned long long *__restrict__ gt,
    unsigned long long *__restrict__ eq, const uint64_t *__restrict__ cand,
    const unsigned long long *__restrict__ gt1) {
    __shared__ uint64_t wave_tot[kHistWaves];
    __shared__ int64_t tile_total;
    __shared__ uint32_t flag;
    const uint32_t t = st->prefix;
    // when every key equal to t is taken (always, without ties), they count with the
    // keys above t and nothing is left for the last workgroup
    const bool all_ties = st->n_last == (unsigned long long)st->k_rem;
    unsigned long long *__restrict__ eqc = all_ties ? gt : eq;
    const int lane = int(threadIdx.x) & (kWave - 1);
    if (!st->overflow) {                                // uniform
        // a wave's 64 candidates come in runs from few rows (each run is one
        // wave-round of the split pass): one atomic per row present and kind
        const uint64_t n = st->n_cand;
        const uint64_t stride = uint64_t(gridDim.x) * kHistThreads;
        const uint64_t first = uint64_t(blockIdx.x) * kHistThreads + threadIdx.x;
        for (uint64_t i0 = first - uint64_t(lane); i0 < n; i0 += stride) {   // wave-uniform
            const uint64_t i = i0 + uint64_t(lane);
            const uint64_t c = i < n ? cand[i] : 0;
            const uint32_t key = uint32_t(c);
            const int32_t r = int32_t(c >> 32);
            const bool g = i < n && key > t, e = i < n && key == t;
            uint64_t todo = __ballot(g || e);
            while (todo) {                              // wave-uniform
                const int l = __ffsll((unsigned long long)todo) - 1;
                const int32_t r0 = __shfl(r, l, kWave);
                const bool same = ((todo >> lane) & 1u) && r == r0;
                const uint64_t ng = __popcll(__ballot(same && g));
                const uint64_t ne = __popcll(__ballot(same && e));
                if (lane == l) {
                    if (all_ties) {
                        atomicAdd(&gt[r0], (unsigned long long)(ng + ne));
                    } else {
                        if (ng) atomicAdd(&gt[r0], (unsigned long long)ng);
                        if (ne) atomicAdd(&eq[r0], (unsigned long long)ne);
                    }
                }
                todo &= ~__ballot(same);
            }
        }
        for (uint64_t r = first; r < uint64_t(M); r += stride)
            if (gt1[r]) atomicAdd(&gt[r], gt1[r]);
    } else {
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
        // flush the previous row's counts when the wave moves on to a new row (all
        // lanes take part in the reduction)
        for_each_key<Bits, ALIGNED>(
            W, ldw, M, N, per_wave, per_wave,
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
    if (last_workgroup(st, &flag) && !all_ties) take_ties(M, st, gt, eq, wave_tot, &tile_total);
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
        st->done = 0;
        st->single = 0;
        st->dlo = 0;
        st->dhi = 0;
    }
}

int64_t align256(int64_t v) { return (v + 255) / 256 * 256; }

// Grid of the passes over W and each wave's share of the padded, flattened W:
// at least one vector per lane (small matrices spread over many CUs: there each
// wave's latency, not bandwidth, sets the time), at most kMaxHistGroups workgroups
// (measured: two per CU, each with half the work, run slower), and few enough
// elements per workgroup (< 2^31) that its 32-bit LDS counters cannot overflow.
struct PrunePartition {
    int groups;
    int64_t per_wave;
};

template <typename Bits> PrunePartition prune_partition(int64_t M, int64_t N) {
    const int64_t total = M * padded_n<Bits>(N);
    const int64_t quantum = int64_t(kWave) * PruneTraits<Bits>::VEC;
    const int64_t per_group_min = quantum * kHistWaves;
    int64_t g = (total + per_group_min - 1) / per_group_min;
    if (g > kMaxHistGroups) g = kMaxHistGroups;
    if (g < 1) g = 1;
    while (g * (int64_t(1) << 30) < total) g *= 2;
    const int64_t waves = g * kHistWaves;
    int64_t per_wave = (total + waves - 1) / waves;
    per_wave = (per_wave + quantum - 1) / quantum * quantum;
    return {int(g), per_wave};
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
                          int64_t *counts, void *workspace, int64_t cand_room, hipStream_t s) {
    using Tr = PruneTraits<Bits>;
    const Bits *W = static_cast<const Bits *>(Wv);
    const PruneWorkspace w = prune_workspace(M, N, workspace);
    PruneState *st = w.st;
    int64_t *eq = w.eq;
    auto *total_u = reinterpret_cast<unsigned long long *>(w.total);
    const PrunePartition part = prune_partition<Bits>(M, N);
    const int groups = part.groups;
    const int64_t per_wave = part.per_wave;
    const int64_t init_n = M > (int64_t(1) << kMaxDigitBits) ? M : (int64_t(1) << kMaxDigitBits);
    const int64_t init_blocks = (init_n + 255) / 256;
    if (init_blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    // the split pass pays for its extra launches only on large matrices: below
    // kSplitMinBytes of W every pass streams W
    const int split = M * N * int64_t(sizeof(Bits)) >= kSplitMinBytes ? 1 : 0;
    hipLaunchKernelGGL(prune_init_kernel, dim3(unsigned(init_blocks)), dim3(256), 0, s, M, k, st,
                       counts, eq, w.gt1, w.total, split);
    if (k == 0) return hipGetLastError();               // nothing kept: counts stay 0

    const bool aligned = (reinterpret_cast<uintptr_t>(W) % 16 == 0) &&
                         ((ldw * int64_t(sizeof(Bits))) % 16 == 0);
    // digit widths from the most significant end
    const int widths32[3] = {11, 10, 10}, widths16[2] = {8, 7};
    const int *widths = Tr::KEY_BITS == 31 ? widths32 : widths16;
    const int passes = Tr::KEY_BITS == 31 ? 3 : 2;
    const uint64_t cap = uint64_t(cand_room);
    auto *gt1_u = reinterpret_cast<unsigned long long *>(w.gt1);
    // more predicted candidates than this and the sample's bracket is not used
    const uint64_t cand_limit =
        std::min<uint64_t>(cap / 2, uint64_t(groups) * uint64_t(kSplitLds) / 2);
    auto hist = [&](int grid, int64_t pw, int64_t stride, int shift, int width, int from_cand,
                    int role) {
        if (aligned)
            hipLaunchKernelGGL((prune_hist_kernel<Bits, true>), dim3(grid), dim3(kHistThreads),
                               0, s, W, ldw, M, N, pw, stride, shift, width, st, total_u, w.cand,
                               from_cand, role, cand_limit);
        else
            hipLaunchKernelGGL((prune_hist_kernel<Bits, false>), dim3(grid), dim3(kHistThreads),
                               0, s, W, ldw, M, N, pw, stride, shift, width, st, total_u, w.cand,
                               from_cand, role, cand_limit);
    };
    int hi = Tr::KEY_BITS;
    for (int p = 0; p < passes; ++p) {
        const int width = widths[p];
        const int shift = hi - width;
        if (p == 0 && split) {
            // the sample (one vector per lane out of about every kSampleEvery, the
            // stride drifting by an odd number of vectors so that it does not follow
            // power-of-two rows) proposes the bracket; the full first-digit
            // histogram runs only when the bracket would hold too many candidates;
            // the split pass then reads W once
            const int64_t chunk = kSampleChunk * int64_t(kWave) * Tr::VEC;
            hist(std::min(groups, kSampleGroups), chunk,
                 kSampleEvery * chunk + kSampleDrift * Tr::VEC, shift, width, 0, kRoleSample);
            hist(groups, per_wave, per_wave, shift, width, 0, kRoleFirst);
            if (aligned)
                hipLaunchKernelGGL((prune_split_kernel<Bits, true>), dim3(groups),
                                   dim3(kHistThreads), 0, s, W, ldw, M, N, per_wave, shift, width,
                                   st, gt1_u, w.cand, cap, total_u);
            else
                hipLaunchKernelGGL((prune_split_kernel<Bits, false>), dim3(groups),
                                   dim3(kHistThreads), 0, s, W, ldw, M, N, per_wave, shift, width,
                                   st, gt1_u, w.cand, cap, total_u);
        } else {
            hist(groups, per_wave, per_wave, shift, width, p > 0, kRoleDigit);
        }
        hi = shift;
    }
    auto *gt_u = reinterpret_cast<unsigned long long *>(counts);
    auto *eq_u = reinterpret_cast<unsigned long long *>(eq);
    if (aligned)
        hipLaunchKernelGGL((prune_count_kernel<Bits, true>), dim3(groups), dim3(kHistThreads), 0,
                           s, W, ldw, M, N, per_wave, st, gt_u, eq_u, w.cand, gt1_u);
    else
        hipLaunchKernelGGL((prune_count_kernel<Bits, false>), dim3(groups), dim3(kHistThreads), 0,
                           s, W, ldw, M, N, per_wave, st, gt_u, eq_u, w.cand, gt1_u);
    return hipGetLastError();
}

}  // namespace

int64_t prune_workspace_bytes(int64_t M, int64_t N, int wdtype) {
    (void)wdtype;
    return prune_offsets(M, N).bytes;
}

hipError_t launch_prune_counts(int64_t M, int64_t N, int wdtype, const void *W, int64_t ldw,
                               int64_t k, int64_t *counts, void *workspace, hipStream_t s) {
    const int64_t room = cand_capacity(M, N);
    if (wdtype == DARB_F32)
        return launch_prune_t<uint32_t>(M, N, W, ldw, k, counts, workspace, room, s);
    return launch_prune_t<uint16_t>(M, N, W, ldw, k, counts, workspace, room, s);
}

// ---------------------------------------------------------------------------------
// The same pruning with its workspace in a fixed device array, for callers that
// cannot allocate.  Every call on a device shares that device's array (the init
// kernel clears what must start at zero on each call), so calls that overlap on one
// device race.  The array holds the radix-select state, the digit totals, the two
// per-row counters (16 bytes per row) and a candidate room of whatever is left,
// never less than kStaticMinRoom keys; a smaller room than the allocating call's
// only sends more of the later passes back to W (same counts).
// ---------------------------------------------------------------------------------

namespace {
constexpr int64_t kStaticScratchBytes = int64_t(8) << 20;
constexpr int64_t kStaticMinRoom = int64_t(1) << 16;
constexpr int kMaxDevices = 64;
}  // namespace

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

int64_t prune_static_max_rows() {
    const PruneOffsets o = prune_offsets(1, 1);
    // fixed part, then 2 x align256(8 M) of row counters, then the minimum room
    const int64_t fixed = o.eq;
    const int64_t avail = kStaticScratchBytes - fixed - kStaticMinRoom * int64_t(sizeof(uint64_t));
    return avail / (2 * int64_t(sizeof(int64_t))) / 32 * 32;   // keeps each counter 256-aligned
}

// The device address of `scratch` on the current device, looked up once per device
// (each device holds its own copy of the array at its own address).
static hipError_t static_scratch(void **ptr) {
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t launch_prune_counts_static(int64_t M, int64_t N, int wdtype, const void *W,
                                      int64_t ldw, int64_t k, int64_t *counts, hipStream_t s) {
    void *ws = nullptr;
    const hipError_t e = static_scratch(&ws);
    if (e != hipSuccess) return e;
    const PruneOffsets o = prune_offsets(M, N);
    const int64_t avail = (kStaticScratchBytes - o.cand) / int64_t(sizeof(uint64_t));
    const int64_t full = cand_capacity(M, N);
    if (avail < full && avail < kStaticMinRoom) return hipErrorInvalidValue;   // caller checked M
    const int64_t room = avail < full ? avail : full;
    if (wdtype == DARB_F32)
        return launch_prune_t<uint32_t>(M, N, W, ldw, k, counts, ws, room, s);
    return launch_prune_t<uint16_t>(M, N, W, ldw, k, counts, ws, room, s);
}

}  // namespace darb
