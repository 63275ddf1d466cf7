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
// proposes a bracket of finer first digits (the key's top 14 bits for fp32, 11 for
// fp16: a bracket as narrow as the sample's statistics allow, not the width of one
// 11-bit digit) that holds the K-th key's, with a margin of six binomial standard
// deviations.  The split pass then counts, per row, the keys whose first digit is
// above the bracket (and their total, G) and copies the keys
// inside it -- the candidates, typically about 1 % of W -- with their rows into the
// workspace.  If G < K <= G + (candidates), the K-th key is a candidate: the
// remaining selection runs over the candidates' keys relative to the bracket's
// lowest key (17 + log2(bracket digits) bits for fp32), for the K - G-th
// largest, and the final counts add the candidates above the threshold to the
// per-row counts above the bracket.  Each workgroup gathers its candidates in LDS
// and reserves room for them with one atomic; if a workgroup's LDS or the
// workspace's candidate room overflows, or the K-th key lies outside the bracket,
// the later passes stream W from the first digit on instead (the result is the
// same).  When the sample predicts more candidates than half the room, the split
// pass takes the exact first-digit histogram of W instead, and the later passes
// stream W for the remaining digits.  The host launches as many passes after the
// split as the digits of the key need; a pass that finds every bit chosen ends at
// once.  Below 64 MiB of W there is no sample and no split: every pass streams W,
// which there costs less than the extra launches.
//
// A pass over the candidates runs as many workgroups as they fill; only those take
// part in finding the last workgroup (a device-wide counter that every
// participating workgroup increments: 256 increments of one address cost about
// 2 us on this chip, and so do 256 workgroups adding their bins into the same
// totals).  The final count needs no last workgroup unless the threshold key has
// ties that only some of its copies are kept for.
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

// Radix-select state, in the workspace.  The keys a pass looks at are taken
// relative to `base` (0, or the bracket's lowest key when the candidates hold the
// threshold): rel = key - base; the digits chosen so far are rel >> hi.
struct PruneState {
    uint32_t prefix;        // the digits chosen so far; with hi = 0, the threshold's rel
    uint32_t hi;            // low bits of rel still to choose (0: the threshold is known)
    uint32_t base;          // subtracted from every key
    uint32_t from_cand;     // every key that matches the prefix is among the candidates
    uint32_t overflow;      // some workgroup's candidates did not fit
    uint32_t done;          // workgroups finished in the running pass (0 between passes)
    uint32_t single;        // the split pass keeps the sample's bracket
    uint32_t dlo, dhi;      // first digits the split pass keeps as candidates
    uint32_t pad;
    int64_t k_rem;          // keys still to take at or below the prefix
    unsigned long long n_cand;   // candidates stored
    unsigned long long n_above;  // keys whose first digit is above the bracket
    unsigned long long n_last;   // keys matching the prefix after the latest digit
};

// What one histogram pass selects: the keys with (key - base) >> hi == prefix,
// by their next digit, for the k_rem-th largest; from the candidates or from W.
struct Pass {
    uint32_t prefix, hi, base;
    bool cand;
    int64_t k_rem;
};

// Width of the next digit when `hi` bits remain: at most kMaxDigitBits, and two
// near-equal digits when two suffice (31 bits: 11, 10, 10; 15 bits: 8, 7).
__host__ __device__ constexpr int digit_width(int hi) {
    return hi > 2 * kMaxDigitBits ? kMaxDigitBits : hi > kMaxDigitBits ? (hi + 1) / 2 : hi;
}
__host__ __device__ constexpr int digit_passes(int hi) {
    return hi <= 0 ? 0 : 1 + digit_passes(hi - digit_width(hi));
}

constexpr int kSplitLds = 8192;                     // candidates a workgroup can hold
constexpr int kWaveRoom = kSplitLds / (1024 / 64);  // of which each of its waves' own
constexpr int64_t kSampleEvery = 32;                // the sample reads about 1/32 of W
constexpr int64_t kSampleDrift = 37;                // vectors added to the sample stride
constexpr int64_t kSampleChunk = 4;                 // vectors per lane in one sampled range
constexpr int kSampleGroups = 256;                  // workgroups of the sample pass
constexpr int kCandPerThread = 8;                   // candidate passes: keys per thread
constexpr int64_t kSplitMinBytes = int64_t(64) << 20;   // W size from which the split pays

template <typename Bits> struct PruneTraits;
template <> struct PruneTraits<uint32_t> {
    static constexpr int VEC = 4;
    static constexpr int UNROLL = 4;        // 16-byte loads per lane per round
    static constexpr int KEY_BITS = 31;
    static constexpr int SAMPLE_BITS = 14;  // the sample's and split's first digit
    static constexpr uint32_t MAG = 0x7FFFFFFFu;
};
template <> struct PruneTraits<uint16_t> {
    static constexpr int VEC = 8;
    static constexpr int UNROLL = 2;        // 16 keys per lane per round (32 measured slower)
    static constexpr int KEY_BITS = 15;
    static constexpr int SAMPLE_BITS = 11;
    static constexpr uint32_t MAG = 0x7FFFu;
};
// The sample's totals of its finer first digit, in the workspace.
constexpr int kFineBins = 1 << 14;

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

// Called by every thread of a workgroup after its global atomics, in the first
// `active` workgroups of the grid (the others take no part in the pass): true in
// the one workgroup that finishes the pass last, which also clears the counter for
// the next pass.  Every value that crosses workgroups goes through device-wide
// read-modify-write atomics, which are coherent across the chip's L2 caches: each
// thread waits until its own atomics are acknowledged before the barrier, so they
// precede the workgroup's increment of the counter, and the last workgroup reads
// the totals with read-modify-write atomics too.  (An agent-scope fence would
// write back and invalidate the L2 in every wave of every workgroup.)
__device__ __forceinline__ bool last_workgroup(PruneState *st, uint32_t *flag, uint32_t active) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t before = atomicAdd(&st->done, 1u);
        const bool last = before == active - 1;
        if (last) atomicExch(&st->done, 0u);
        *flag = last ? 1u : 0u;
    }
    __syncthreads();
    return *flag != 0;
}

// One workgroup, after a histogram pass P with a digit of `width` bits: find the
// digit d where the count of matching keys with digit > d is < k_rem <= that count
// plus total[d], append it to the prefix, and clear `total` for the next pass.
// Writes the whole selection (the pass may have derived base and source itself).
__device__ __forceinline__ void select_digit(unsigned long long *__restrict__ total,
                                             const Pass &P, int width,
                                             PruneState *__restrict__ st, uint64_t *tot,
                                             uint64_t *wave_tot) {
    const int bins = 1 << width;
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) tot[b] = atomicExch(&total[b], 0ull);
    __syncthreads();
    // thread t owns the digits bins-1-2t and bins-2-2t (descending order)
    const int d0 = bins - 1 - 2 * int(threadIdx.x), d1 = d0 - 1;
    const uint64_t a = d0 >= 0 ? tot[d0] : 0, b = d1 >= 0 ? tot[d1] : 0;
    const uint64_t incl = block_inclusive_scan(a + b, wave_tot);
    const uint64_t excl = incl - a - b;
    const uint64_t k = uint64_t(P.k_rem);
    if (threadIdx.x == 0) {
        st->hi = P.hi - uint32_t(width);
        st->base = P.base;
        st->from_cand = P.cand ? 1u : 0u;
    }
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
        st->prefix = (P.prefix << width) | d;
        st->k_rem = int64_t(k - above);
        st->n_last = d == uint32_t(d0) ? a : b;
    }
}

// One workgroup, after the sample (n_s keys out of the matrix's total_keys, a
// fraction f): the split pass's bracket [dlo, dhi] of fine first digits (the top FB
// bits of the key) that holds the k-th largest key's, up to six standard
// deviations of the sample count (a binomial) plus 8 keys: keys above dhi number
// at most f*k - margin in the sample, keys at or above dlo at least f*k + margin.
// One pass over W then suffices (`single`) unless the bracket's predicted
// candidates exceed cand_limit.  The sample's totals are kept per coarse digit (the
// top CB bits, in `total`, which this clears for the next pass) and per fine
// digit (in `fine`, zeroed by the state reset): the coarse totals place the two
// ends within a coarse digit each, and only those digits' fine totals are read
// (reading every fine total from one workgroup costs about 10 us).
template <int CB_BITS, int FB_BITS>
__device__ __forceinline__ void select_bracket(unsigned long long *__restrict__ total,
                                               unsigned long long *__restrict__ fine,
                                               PruneState *__restrict__ st, int64_t total_keys,
                                               int64_t k, uint64_t cand_limit, uint64_t *tot,
                                               uint64_t *wave_tot, uint32_t *s_d, uint64_t *s_c,
                                               uint64_t *s_f) {
    constexpr int CB = 1 << CB_BITS;
    constexpr int R = 1 << (FB_BITS - CB_BITS);         // fine digits per coarse digit
    constexpr uint32_t kNone = 0xFFFFFFFFu;
    static_assert(2 * R <= kHistThreads, "one thread per boundary fine digit");
    for (int b = int(threadIdx.x); b < CB; b += kHistThreads) tot[b] = atomicExch(&total[b], 0ull);
    if (threadIdx.x == 0) {
        s_d[0] = kNone;                                 // coarse digit of dhi
        s_d[1] = kNone;                                 // coarse digit of dlo
    }
    __syncthreads();
    // thread t owns the coarse digits CB-1-2t and CB-2-2t (descending order)
    const int d0 = CB - 1 - 2 * int(threadIdx.x), d1 = d0 - 1;
    const uint64_t a = d0 >= 0 ? tot[d0] : 0, b = d1 >= 0 ? tot[d1] : 0;
    const uint64_t incl = block_inclusive_scan(a + b, wave_tot);
    const uint64_t excl = incl - a - b;
    if (threadIdx.x == kHistThreads - 1) s_c[4] = incl;
    __syncthreads();
    const uint64_t n_s = s_c[4];
    const double q = double(k) / double(total_keys);
    const double ks = q * double(n_s);
    const double margin = 6.0 * sqrt(ks * (1.0 - q)) + 8.0;
    const double lo = ks - margin, hi = ks + margin;
    // digit d has `above` keys with a larger digit and `above + c` at or above it,
    // both non-increasing in d: dhi is the one digit with above <= lo < above + c
    // (or digit 0 with above <= lo), dlo the one with above < hi <= above + c (or
    // the top digit with above + c >= hi); first among the coarse digits
    auto coarse = [&](int d, uint64_t above, uint64_t c) {
        if (d < 0) return;
        const double ab = double(above), at = double(above + c);
        if (ab <= lo && (d == 0 || at > lo)) {
            s_d[0] = uint32_t(d);
            s_c[0] = above;
            s_c[1] = c;
        }
        if (at >= hi && (d == CB - 1 || ab < hi)) {
            s_d[1] = uint32_t(d);
            s_c[2] = above;
            s_c[3] = c;
        }
    };
    coarse(d0, excl, a);
    coarse(d1, excl + a, b);
    __syncthreads();
    const uint32_t chi = s_d[0], clo = s_d[1];
    // then among the fine digits of those two coarse digits
    if (threadIdx.x < 2 * R) {
        const uint32_t c = threadIdx.x < R ? chi : clo;
        s_f[threadIdx.x] =
            c == kNone ? 0ull : atomicAdd(&fine[c * R + (threadIdx.x & (R - 1))], 0ull);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        constexpr uint32_t kTop = (1u << FB_BITS) - 1;
        // defaults: the whole range at an end no digit qualifies for, the whole
        // coarse digit if its fine totals disagree with it
        uint32_t dhi = kTop, dlo = 0;
        uint64_t above_hi = 0, at_lo = n_s;
        if (chi != kNone) {
            dhi = chi * R + R - 1;
            above_hi = s_c[0];
            uint64_t ab = s_c[0];
            for (int j = R - 1; j >= 0; --j) {
                const uint32_t f = chi * R + uint32_t(j);
                if (double(ab) <= lo && (f == 0 || double(ab + s_f[j]) > lo)) {
                    dhi = f;
                    above_hi = ab;
                    break;
                }
                ab += s_f[j];
            }
        }
        if (clo != kNone) {
            dlo = clo * R;
            at_lo = s_c[2] + s_c[3];
            uint64_t ab = s_c[2];
            for (int j = R - 1; j >= 0; --j) {
                const uint32_t f = clo * R + uint32_t(j);
                if (double(ab + s_f[R + j]) >= hi) {
                    dlo = f;
                    at_lo = ab + s_f[R + j];
                    break;
                }
                ab += s_f[R + j];
            }
        }
        // predicted candidates: the bracket's sample keys scaled by 1/f
        const bool ok = dlo <= dhi && at_lo >= above_hi;
        const uint64_t in_all = ok ? at_lo - above_hi : 0;
        const bool fits = ok && n_s > 0 && double(in_all) * double(total_keys) <=
                                               double(cand_limit) * double(n_s);
        st->single = fits ? 1u : 0u;
        st->dlo = dlo;
        st->dhi = dhi;
    }
}

// What a histogram pass is for.
enum HistRole {
    kRoleNext = 0,        // the next digit, as the state describes it
    kRoleAfterSplit = 1,  // the first pass after the split: from the candidates if they
                          // hold the threshold, else from W (from the first digit on)
};

// Number of bits needed to write v (0 for 0).
__device__ __forceinline__ uint32_t bit_length(uint32_t v) { return v ? 32u - __clz(v) : 0u; }

// The pass the state describes; for the first pass after a split pass that kept
// the sample's bracket, the one its results call for (every workgroup derives the
// same from the same state): the candidates' keys relative to the bracket's lowest
// key when G < k <= G + candidates (G the keys above the bracket), else all of W
// from the first digit.  `cap` bounds the candidate count read from the state.
template <typename Bits>
__device__ __forceinline__ Pass pass_from_state(const PruneState *__restrict__ st, int role,
                                                int64_t k, uint64_t cap) {
    constexpr int KB = PruneTraits<Bits>::KEY_BITS;
    Pass P;
    if (role == kRoleAfterSplit && st->single) {
        constexpr int first_shift = KB - PruneTraits<Bits>::SAMPLE_BITS;
        const uint64_t G = st->n_above, n = st->n_cand, kk = uint64_t(k);
        const uint32_t dlo = st->dlo, dhi = st->dhi;
        if (!st->overflow && n <= cap && dlo <= dhi && G < kk && kk <= G + n) {
            P.base = dlo << first_shift;
            P.prefix = 0;
            P.hi = uint32_t(first_shift) + bit_length(dhi - dlo);
            P.cand = true;
            P.k_rem = int64_t(kk - G);
        } else {
            P.base = 0;
            P.prefix = 0;
            P.hi = KB;
            P.cand = false;
            P.k_rem = k;
        }
    } else {
        P.base = st->base;
        P.prefix = st->prefix;
        P.hi = st->hi < uint32_t(KB) ? st->hi : uint32_t(KB);
        P.cand = st->from_cand != 0;
        P.k_rem = st->k_rem;
    }
    return P;
}

// One workgroup's part of histogram pass P (digit of `width` bits): the LDS
// histogram of its keys that match the prefix, added into `total`; the keys come
// from W (ranges of per_wave elements range_stride apart) or from the n
// candidates.  Over candidates only the workgroups they fill take part (returns
// false at once in the others).  True in the workgroup that finishes last.
template <typename Bits, bool ALIGNED>
__device__ __forceinline__ bool hist_pass(const Bits *__restrict__ W, int64_t ldw, int64_t M,
                                          int64_t N, int64_t per_wave, int64_t range_stride,
                                          const Pass &P, int width, uint64_t n,
                                          PruneState *__restrict__ st,
                                          unsigned long long *__restrict__ total,
                                          const uint64_t *__restrict__ cand, uint32_t *hist,
                                          uint32_t *flag) {
    constexpr int kStride = (1 << kMaxDigitBits) + 1;   // copies land in different banks
    const int bins = 1 << width;
    // kCandPerThread candidates per thread: few workgroups, so few bins to flush
    const uint64_t per_group = uint64_t(kCandPerThread) * kHistThreads;
    uint32_t active = gridDim.x;
    if (P.cand) {
        const uint64_t g = n > per_group ? (n + per_group - 1) / per_group : 1;
        if (g < active) active = uint32_t(g);
    }
    if (blockIdx.x >= active) return false;            // uniform
    // over candidates, the thread's first keys are on their way while the histogram
    // is cleared (the barrier waits for the LDS writes only)
    const uint64_t stride = uint64_t(active) * kHistThreads;
    uint64_t i0 = uint64_t(blockIdx.x) * kHistThreads + threadIdx.x;
    uint32_t kk[kCandPerThread];
    auto load_batch = [&]() {
#pragma unroll
        for (int j = 0; j < kCandPerThread; ++j) {
            const uint64_t i = i0 + uint64_t(j) * stride;
            kk[j] = i < n ? uint32_t(cand[i]) : 0u;
        }
    };
    if (P.cand) load_batch();
    for (int i = int(threadIdx.x); i < kCopies * kStride; i += kHistThreads) hist[i] = 0;
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    const uint32_t prefix = P.prefix, base = P.base, hi = P.hi;   // hi <= key bits <= 31
    const uint32_t shift = hi - uint32_t(width);
    const uint32_t dmask = uint32_t(bins - 1);
    uint32_t *mine = hist + (int(threadIdx.x) & (kCopies - 1)) * kStride;
    auto add = [&](uint32_t key) {
        const uint32_t rel = key - base;
        if ((rel >> hi) == prefix) atomicAdd(&mine[(rel >> shift) & dmask], 1u);
    };
    if (P.cand) {
        // all of a batch's loads issued before its LDS atomics
        while (i0 < n) {
#pragma unroll
            for (int j = 0; j < kCandPerThread; ++j)
                if (i0 + uint64_t(j) * stride < n) add(kk[j]);
            i0 += stride * kCandPerThread;
            if (i0 < n) load_batch();
        }
    } else {
        for_each_key<Bits, ALIGNED>(W, ldw, M, N, per_wave, range_stride, [](int64_t) {}, add);
    }
    __syncthreads();
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) {
        uint32_t s = 0;
#pragma unroll
        for (int c = 0; c < kCopies; ++c) s += hist[c * kStride + b];
        if (s) atomicAdd(&total[b], (unsigned long long)s);
    }
    return last_workgroup(st, flag, active);
}

// A histogram pass (role above); the last workgroup picks the digit.  A pass that
// finds every bit chosen does nothing.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_hist_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave,
    int64_t range_stride, PruneState *__restrict__ st, unsigned long long *__restrict__ total,
    const uint64_t *__restrict__ cand, int role, int64_t k, uint64_t cap) {
    constexpr int kStride = (1 << kMaxDigitBits) + 1;
    __shared__ uint32_t hist[kCopies * kStride];
    __shared__ uint64_t tot[1 << kMaxDigitBits];
    __shared__ uint64_t wave_tot[kHistWaves];
    __shared__ uint32_t flag;
    const Pass P = pass_from_state<Bits>(st, role, k, cap);
    if (P.hi == 0) return;                              // uniform: the threshold is known
    const int width = digit_width(int(P.hi));
    uint64_t n = 0;
    if (P.cand) {
        n = st->n_cand;
        if (n > cap) n = cap;
    }
    if (!hist_pass<Bits, ALIGNED>(W, ldw, M, N, per_wave, range_stride, P, width, n, st, total,
                                  cand, hist, &flag))
        return;
    select_digit(total, P, width, st, tot, wave_tot);
}

// The sample: the histogram of the keys' first SAMPLE_BITS bits over ranges of
// chunk elements range_stride apart (one range per wave), added into `fine`, and
// of their first digit_width(KEY_BITS) bits, added into `total`; the last
// workgroup picks the split pass's bracket.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_sample_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t chunk,
    int64_t range_stride, PruneState *__restrict__ st, unsigned long long *__restrict__ total,
    unsigned long long *__restrict__ fine, int64_t k, uint64_t cand_limit) {
    constexpr int KB = PruneTraits<Bits>::KEY_BITS;
    constexpr int FB = PruneTraits<Bits>::SAMPLE_BITS;
    constexpr int CB = digit_width(KB);
    constexpr int R = 1 << (FB - CB);
    constexpr uint32_t shift = uint32_t(KB - FB);
    __shared__ uint32_t hist[1 << FB];
    __shared__ uint64_t tot[1 << CB];
    __shared__ uint64_t wave_tot[kHistWaves];
    __shared__ uint64_t s_c[5], s_f[2 * R];
    __shared__ uint32_t s_d[2], flag;
    for (int i = int(threadIdx.x); i < (1 << FB); i += kHistThreads) hist[i] = 0;
    __syncthreads();
    for_each_key<Bits, ALIGNED>(W, ldw, M, N, chunk, range_stride, [](int64_t) {},
                                [&](uint32_t key) { atomicAdd(&hist[key >> shift], 1u); });
    __syncthreads();
    for (int b = int(threadIdx.x); b < (1 << FB); b += kHistThreads) {
        const uint32_t v = hist[b];
        if (v) atomicAdd(&fine[b], (unsigned long long)v);
    }
    for (int c = int(threadIdx.x); c < (1 << CB); c += kHistThreads) {
        uint32_t v = 0;
#pragma unroll
        for (int j = 0; j < R; ++j) v += hist[c * R + j];
        if (v) atomicAdd(&total[c], (unsigned long long)v);
    }
    if (!last_workgroup(st, &flag, gridDim.x)) return;
    select_bracket<CB, FB>(total, fine, st, M * N, k, cand_limit, tot, wave_tot, s_d, s_c, s_f);
}

// The split pass, once the sample's bracket [dlo, dhi] of first digits is known:
// per row, the keys with first digit > dhi go to gt1 (and their total to the
// state's n_above); keys with first digit in the bracket are stored as
// (row << 32 | key) candidates.  Runs in the same grid as the histogram passes.  If
// any workgroup's candidates overflow its LDS or the workspace's room, the state's
// overflow flag sends the later passes back to W.  Without `single` (the bracket
// would hold too many keys) it takes the exact first digit over W instead.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_split_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave,
    PruneState *__restrict__ st, unsigned long long *__restrict__ gt1,
    uint64_t *__restrict__ cand, uint64_t cap, unsigned long long *__restrict__ total) {
    constexpr int kStride = (1 << kMaxDigitBits) + 1;
    constexpr int KB = PruneTraits<Bits>::KEY_BITS;
    constexpr int first_shift = KB - PruneTraits<Bits>::SAMPLE_BITS;
    __shared__ uint64_t buf[kSplitLds];
    __shared__ uint32_t hist[kCopies * kStride];
    __shared__ uint64_t tot[1 << kMaxDigitBits];
    __shared__ uint64_t wave_tot[kHistWaves];
    __shared__ uint32_t wave_n[kHistWaves], flag;
    __shared__ uint64_t base;
    if (!st->single) {                                  // uniform
        Pass P;
        P.prefix = 0;
        P.hi = KB;
        P.base = 0;
        P.cand = false;
        P.k_rem = st->k_rem;
        if (hist_pass<Bits, ALIGNED>(W, ldw, M, N, per_wave, per_wave, P, digit_width(KB), 0, st,
                                     total, cand, hist, &flag))
            select_digit(total, P, digit_width(KB), st, tot, wave_tot);
        return;
    }
    static_assert(kWaveRoom * kHistWaves == kSplitLds, "one LDS region per wave");
    const uint32_t dlo = st->dlo, dhi = st->dhi;
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
    uint64_t *mine = buf + wave * kWaveRoom;
    // the wave's candidates so far and its keys above the bracket (wave-uniform):
    // each wave fills its own LDS region, so no atomic (and no wait for one) sits
    // between a round's keys and the next round's loads
    uint32_t wn = 0;
    uint64_t w_above = 0;
    int64_t cur = -1;
    uint32_t n_gt = 0;
    auto flush = [&]() {
        uint32_t g = n_gt;
#pragma unroll
        for (int m = kWave / 2; m >= 1; m >>= 1) g += __shfl_xor(g, m, kWave);
        if (lane == 0 && cur >= 0 && g) atomicAdd(&gt1[cur], (unsigned long long)g);
        w_above += g;
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
            // mask of the candidates; then one ballot per key slot, and each lane
            // places its own candidates by the set bits below it in the ballot
            uint32_t cm = 0;
#pragma unroll
            for (int j = 0; j < K; ++j) {
                const uint32_t top = keys[j] >> first_shift;
                const bool in = (mask >> j) & 1u;
                n_gt += (in && top > dhi) ? 1u : 0u;
                cm |= (in && top >= dlo && top <= dhi) ? (1u << j) : 0u;
            }
#pragma unroll
            for (int j = 0; j < K; ++j) {
                const uint64_t bal = __ballot((cm >> j) & 1u);
                if (bal) {                              // wave-uniform
                    const uint32_t p = wn + __builtin_amdgcn_mbcnt_hi(
                                                 uint32_t(bal >> 32),
                                                 __builtin_amdgcn_mbcnt_lo(uint32_t(bal), 0u));
                    if (((cm >> j) & 1u) && p < uint32_t(kWaveRoom))
                        mine[p] = (uint64_t(cur) << 32) | keys[j];
                    wn += uint32_t(__popcll(bal));
                }
            }
        });
    flush();
    if (lane == 0) {
        wave_n[wave] = wn;
        wave_tot[wave] = w_above;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t n = 0;
        bool over = false;
        uint64_t above = 0;
        for (int w = 0; w < kHistWaves; ++w) {
            n += wave_n[w];
            over = over || wave_n[w] > uint32_t(kWaveRoom);
            above += wave_tot[w];
        }
        uint64_t b = 0;
        if (over) {
            atomicExch(&st->overflow, 1u);
            b = cap;                                    // nothing is copied
        } else if (n > 0) {
            b = atomicAdd(&st->n_cand, (unsigned long long)n);
            if (b + n > cap) {
                atomicExch(&st->overflow, 1u);
                b = cap;
            }
        }
        if (above) atomicAdd(&st->n_above, (unsigned long long)above);
        base = b;
    }
    __syncthreads();
    if (base < cap) {                                   // uniform: the room was reserved
        uint64_t at = base;
        for (int w = 0; w < wave; ++w) at += wave_n[w];
        for (uint32_t i = uint32_t(lane); i < wn; i += kWave) cand[at + i] = mine[i];
    }
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

// Per-row counts of keys > t (into counts) and == t (into eq); t = base + prefix.
// From the candidates when they hold the threshold (plus the split pass's gt1),
// else from W.  When only some keys == t are kept, the last workgroup to finish
// then adds those.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_count_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave,
    PruneState *__restrict__ st, unsigned long long *__restrict__ gt,
    unsigned long long *__restrict__ eq, const uint64_t *__restrict__ cand,
    const unsigned long long *__restrict__ gt1, uint64_t cap) {
    __shared__ uint64_t wave_tot[kHistWaves];
    __shared__ int64_t tile_total;
    __shared__ uint32_t flag;
    const uint32_t t = st->base + st->prefix;
    // when every key equal to t is taken (always, without ties), they count with the
    // keys above t and nothing is left for the last workgroup
    const bool all_ties = st->n_last == (unsigned long long)st->k_rem;
    unsigned long long *__restrict__ eqc = all_ties ? gt : eq;
    const int lane = int(threadIdx.x) & (kWave - 1);
    if (st->from_cand) {                                // uniform
        // a wave's 64 candidates come in runs from few rows (each run is one
        // wave-round of the split pass): one atomic per row present and kind
        uint64_t n = st->n_cand;
        if (n > cap) n = cap;
        const uint64_t stride = uint64_t(gridDim.x) * kHistThreads;
        const uint64_t first = uint64_t(blockIdx.x) * kHistThreads + threadIdx.x;
        for (uint64_t i0 = first - uint64_t(lane); i0 < n; i0 += stride) {   // wave-uniform
            const uint64_t i = i0 + uint64_t(lane);
            const uint64_t c = i < n ? cand[i] : 0;
            const uint32_t key = uint32_t(c);
            const int64_t r = int64_t(c >> 32);
            const bool ok = i < n && r < M;
            const bool g = ok && key > t, e = ok && key == t;
            uint64_t todo = __ballot(g || e);
            while (todo) {                              // wave-uniform
                const int l = __ffsll((unsigned long long)todo) - 1;
                const int64_t r0 = __shfl(r, l, kWave);
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
    if (all_ties) return;                               // uniform
    if (last_workgroup(st, &flag, gridDim.x)) take_ties(M, st, gt, eq, wave_tot, &tile_total);
}

// Zero counts, eq, gt1, the digit totals and the sample's fine totals, and set the state to (no digit
// chosen: prefix 0, hi = the key's bits, base 0; k_rem = k, no candidates).
__global__ __launch_bounds__(256) void prune_init_kernel(int64_t M, int64_t k, int key_bits,
                                                         PruneState *st, int64_t *counts,
                                                         int64_t *eq, int64_t *gt1,
                                                         uint64_t *total, uint64_t *fine) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i < M) {
        counts[i] = 0;
        eq[i] = 0;
        gt1[i] = 0;
    }
    if (i < (int64_t(1) << kMaxDigitBits)) total[i] = 0;
    if (i < kFineBins) fine[i] = 0;
    if (i == 0 && st) {
        st->prefix = 0;
        st->hi = uint32_t(key_bits);
        st->base = 0;
        st->from_cand = 0;
        st->overflow = 0;
        st->done = 0;
        st->single = 0;
        st->dlo = 0;
        st->dhi = 0;
        st->pad = 0;
        st->k_rem = k;
        st->n_cand = 0;
        st->n_above = 0;
        st->n_last = 0;
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
    uint64_t *fine;         // [kFineBins]
    int64_t *eq;            // [M]
    int64_t *gt1;           // [M]
    uint64_t *cand;         // [cand_capacity]
};

struct PruneOffsets { int64_t total, fine, eq, gt1, cand, bytes; };

PruneOffsets prune_offsets(int64_t M, int64_t N) {
    PruneOffsets o;
    o.total = align256(int64_t(sizeof(PruneState)));
    o.fine = o.total + align256((int64_t(1) << kMaxDigitBits) * 8);
    o.eq = o.fine + align256(int64_t(kFineBins) * 8);
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
    w.fine = reinterpret_cast<uint64_t *>(c + o.fine);
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
    auto *fine_u = reinterpret_cast<unsigned long long *>(w.fine);
    const PrunePartition part = prune_partition<Bits>(M, N);
    const int groups = part.groups;
    const int64_t per_wave = part.per_wave;
    const int64_t init_n = M > kFineBins ? M : kFineBins;
    const int64_t init_blocks = (init_n + 255) / 256;
    if (init_blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(prune_init_kernel, dim3(unsigned(init_blocks)), dim3(256), 0, s, M, k,
                       int(Tr::KEY_BITS), st, counts, eq, w.gt1, w.total, w.fine);
    if (k == 0) return hipGetLastError();               // nothing kept: counts stay 0

    const bool aligned = (reinterpret_cast<uintptr_t>(W) % 16 == 0) &&
                         ((ldw * int64_t(sizeof(Bits))) % 16 == 0);
    // digits of the whole key (3 for fp32, 2 for fp16): every way through the
    // passes needs at most that many after the first digit's pass or the split
    constexpr int passes = digit_passes(Tr::KEY_BITS);
    const uint64_t cap = uint64_t(cand_room);
    auto *gt1_u = reinterpret_cast<unsigned long long *>(w.gt1);
    // more predicted candidates than this and the split pass takes the first digit
    const uint64_t cand_limit =
        std::min<uint64_t>(cap / 2, uint64_t(groups) * uint64_t(kSplitLds) / 2);
    auto hist = [&](int role) {
        if (aligned)
            hipLaunchKernelGGL((prune_hist_kernel<Bits, true>), dim3(groups), dim3(kHistThreads),
                               0, s, W, ldw, M, N, per_wave, per_wave, st, total_u, w.cand, role,
                               k, cap);
        else
            hipLaunchKernelGGL((prune_hist_kernel<Bits, false>), dim3(groups),
                               dim3(kHistThreads), 0, s, W, ldw, M, N, per_wave, per_wave, st,
                               total_u, w.cand, role, k, cap);
    };
    // the split pass pays for its extra launches only on large matrices: below
    // kSplitMinBytes of W every pass streams W
    if (M * N * int64_t(sizeof(Bits)) >= kSplitMinBytes) {
        // the sample (ranges of kSampleChunk vectors per lane, one out of about every
        // kSampleEvery, the stride drifting by an odd number of vectors so that it
        // does not follow power-of-two rows) proposes the bracket, in as many
        // workgroups as it has ranges for; the split pass then reads W once
        const int64_t chunk = kSampleChunk * int64_t(kWave) * Tr::VEC;
        const int64_t range_stride = kSampleEvery * chunk + kSampleDrift * Tr::VEC;
        const int64_t ranges = (M * padded_n<Bits>(N) + range_stride - 1) / range_stride;
        const int64_t sample_groups =
            std::min<int64_t>(kSampleGroups, (ranges + kHistWaves - 1) / kHistWaves);
        const dim3 sgrid(unsigned(std::max<int64_t>(1, sample_groups)));
        if (aligned)
            hipLaunchKernelGGL((prune_sample_kernel<Bits, true>), sgrid, dim3(kHistThreads), 0, s,
                               W, ldw, M, N, chunk, range_stride, st, total_u, fine_u, k,
                               cand_limit);
        else
            hipLaunchKernelGGL((prune_sample_kernel<Bits, false>), sgrid, dim3(kHistThreads), 0,
                               s, W, ldw, M, N, chunk, range_stride, st, total_u, fine_u, k,
                               cand_limit);
        if (aligned)
            hipLaunchKernelGGL((prune_split_kernel<Bits, true>), dim3(groups), dim3(kHistThreads),
                               0, s, W, ldw, M, N, per_wave, st, gt1_u, w.cand, cap, total_u);
        else
            hipLaunchKernelGGL((prune_split_kernel<Bits, false>), dim3(groups),
                               dim3(kHistThreads), 0, s, W, ldw, M, N, per_wave, st, gt1_u,
                               w.cand, cap, total_u);
        for (int p = 0; p < passes; ++p) hist(p == 0 ? kRoleAfterSplit : kRoleNext);
    } else {
        for (int p = 0; p < passes; ++p) hist(kRoleNext);
    }
    auto *gt_u = reinterpret_cast<unsigned long long *>(counts);
    auto *eq_u = reinterpret_cast<unsigned long long *>(eq);
    if (aligned)
        hipLaunchKernelGGL((prune_count_kernel<Bits, true>), dim3(groups), dim3(kHistThreads), 0,
                           s, W, ldw, M, N, per_wave, st, gt_u, eq_u, w.cand, gt1_u, cap);
    else
        hipLaunchKernelGGL((prune_count_kernel<Bits, false>), dim3(groups), dim3(kHistThreads), 0,
                           s, W, ldw, M, N, per_wave, st, gt_u, eq_u, w.cand, gt1_u, cap);
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
