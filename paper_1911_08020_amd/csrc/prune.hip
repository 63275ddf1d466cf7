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
// pass's own totals buffer).  The next kernel picks the digit where the count from
// the top reaches the remaining K: every one of its workgroups reads the totals
// (the kernel boundary has made them visible) and chooses the same way, so no
// workgroup waits for the others and no read-modify-write reads totals back.
// Finally, per row, the keys > t are counted and the keys == t taken in flat
// order, which for row counts means rows in ascending order (by the count pass's
// last workgroup, only when some keys equal to t are not kept).
//
// From 64 MiB of W one pass streams all of W.  A sample of W (about 1/32) first
// histograms finer first digits (the key's top 14 bits for fp32, 11 for fp16; the
// same launch resets the state, and the count pass leaves the sample's histogram
// at zero for the next call on the workspace), from
// which the split pass's workgroups compute a bracket of them that holds the K-th
// key's, with a margin of six binomial standard deviations: as narrow as the
// sample's statistics allow, not the width of one 11-bit digit.  The split pass
// then counts, per row, the keys whose first digit is above the bracket (and their
// total, G) and copies the keys inside it -- the candidates, typically under 1 % of
// W -- with their rows into the workspace (each wave fills its own LDS region, each
// workgroup reserves room with one atomic).  If G < K <= G + (candidates), the K-th
// key is a candidate: the remaining selection runs over the candidates' keys
// relative to the bracket's lowest key (17 + log2(bracket digits) bits for fp32),
// for the K - G-th largest, and the final counts add the candidates above the
// threshold to the per-row counts above the bracket.  If a wave's region or the
// workspace's room overflows, or the K-th key lies outside the bracket, the later
// passes stream W from the first digit on instead (the result is the same).  When
// the sample predicts more candidates than half the room, the split pass takes the
// exact first-digit histogram of W instead, and the later passes stream W for the
// remaining digits.  The host launches as many passes after the split as the
// key's digits need; a pass with nothing left to choose hands the state on.  Below
// 64 MiB of W there is no sample and no split: a reset launch, then every pass
// streams W, which there costs less than the extra launches.  A pass over the candidates runs only the
// workgroups they fill.  All state stays on the device; nothing returns to the host
// between passes.
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

// Radix-select state, in two slots of the workspace: each kernel reads one and
// its first workgroup writes the other, which the next kernel reads (a kernel never
// writes the slot its own workgroups read).  The keys a pass looks at are taken
// relative to `base` (0, or the bracket's lowest key when the candidates hold the
// threshold): rel = key - base; the digits chosen so far are rel >> hi.  A pass
// leaves its digit's histogram in its own totals buffer, and the kernel after it
// picks the digit (every workgroup of it, the same way) before its own work: no
// workgroup waits for the others to finish, and no read-modify-write reads the
// totals back.
struct PruneState {
    uint32_t prefix;        // the digits chosen so far; with hi = 0, the threshold's rel
    uint32_t hi;            // low bits of rel still to choose (0: the threshold is known)
    uint32_t base;          // subtracted from every key
    uint32_t from_cand;     // every key that matches the prefix is among the candidates
    int64_t k_rem;          // keys still to take at or below the prefix
    unsigned long long n_last;   // keys matching the prefix after the latest digit
    uint32_t pend_width;    // > 0: the next pend_width bits' histogram is pending,
    uint32_t pend_buf;      //      in totals buffer pend_buf
};

// What the split pass leaves for the passes after it (atomics, or its first
// workgroup), and the count's last-workgroup counter.
struct SplitInfo {
    uint32_t overflow;      // some workgroup's candidates did not fit
    uint32_t single;        // the split pass kept the sample's bracket
    uint32_t dlo, dhi;      // the bracket of fine first digits
    unsigned long long n_cand;   // candidates stored (reserved)
    unsigned long long n_above;  // keys whose first digit is above the bracket
    uint32_t done;          // workgroups of the count finished
    uint32_t pad[3];
};

// Totals buffers, one per digit histogram of a call: the split pass's first digit
// (when it takes one), then one per pass after it.  (The sample's totals are kept
// apart, per fine digit.)
constexpr int kDigitBins = 1 << kMaxDigitBits;
constexpr int kTotalsBuffers = 4;
constexpr int kBufSplit = 0, kBufPass0 = 1;

// What one histogram pass selects: the keys with (key - base) >> hi == prefix,
// by their next digit, for the k_rem-th largest; from the candidates or from W.
struct Pass {
    uint32_t prefix, hi, base;
    bool cand;
    int64_t k_rem;
    unsigned long long n_last;
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
constexpr int kWaveRoom = kSplitLds / kHistWaves;   // of which each of its waves' own
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

// As for_each_round for 16-byte aligned rows, with each round handed over in two
// halves, half(keys, valid, first) (first: the index of keys[0] in the round), and
// the next round's loads issued half by half into the registers the current half's
// keys have just left: half of each round's memory latency overlaps the previous
// round's work without a second set of registers.  The loads stay unconditional
// (a round past the piece's end reloads the piece's first vectors and keeps
// nothing), so the compiler waits for exactly the loads a half needs.
template <typename Bits, typename U, typename H>
__device__ __forceinline__ void for_each_round_halves(const Bits *__restrict__ W, int64_t ldw,
                                                      int64_t M, int64_t N, int64_t per_wave,
                                                      U &&on_unit, H &&half) {
    using Tr = PruneTraits<Bits>;
    constexpr int VEC = Tr::VEC;
    constexpr int kUnroll = Tr::UNROLL;
    constexpr int HU = kUnroll / 2;                     // vectors per half
    static_assert(kUnroll % 2 == 0, "two halves per round");
    constexpr int64_t STEP = round_width<Bits>();
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
    const int64_t gw = int64_t(blockIdx.x) * (blockDim.x / kWave) + wave;
    const int64_t tw = int64_t(gridDim.x) * (blockDim.x / kWave);
    const int64_t Np = padded_n<Bits>(N);
    const int64_t total = M * Np;
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    for (int64_t a = gw * per_wave; a < total; a += tw * per_wave) {   // wave-uniform
        const int64_t b = a + per_wave < total ? a + per_wave : total;
        int64_t r = a / Np;
        int64_t c = a - r * Np;
        for (int64_t at = a; at < b; ++r, c = 0) {
            const int64_t c_piece = c + (b - at) < Np ? c + (b - at) : Np;
            const int64_t c_end = c_piece < N ? c_piece : N;
            at += c_piece - c;
            const Bits *row = W + r * ldw;
            on_unit(r);
            if (c >= c_end) continue;
            PVec<Bits, VEC> v[kUnroll];
            uint32_t valid[kUnroll];                    // bit e: element e is inside the row
            // rows are whole 16-byte vectors apart, so the vector holding a row's last
            // element lies inside the row's stride
            auto load = [&](int q, int64_t c0) {
                const int64_t cc = c0 + int64_t(q) * kWave * VEC + int64_t(lane) * VEC;
                const int64_t left = c_end - cc;
                const u32x4 t = __builtin_nontemporal_load(
                    reinterpret_cast<const u32x4 *>(row + (left > 0 ? cc : c)));
                v[q] = __builtin_bit_cast(PVec<Bits, VEC>, t);
                valid[q] = left >= VEC ? (1u << VEC) - 1u : (left > 0 ? (1u << left) - 1u : 0u);
            };
#pragma unroll
            for (int q = 0; q < kUnroll; ++q) load(q, c);
            for (int64_t c0 = c; c0 < c_end; c0 += STEP) {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    uint32_t keys[HU * VEC];
                    uint32_t mask = 0;
#pragma unroll
                    for (int q = 0; q < HU; ++q) {
#pragma unroll
                        for (int e = 0; e < VEC; ++e)
                            keys[q * VEC + e] = uint32_t(v[h * HU + q].e[e]) & Tr::MAG;
                        mask |= valid[h * HU + q] << (q * VEC);
                    }
#pragma unroll
                    for (int q = 0; q < HU; ++q) load(h * HU + q, c0 + STEP);
                    half(keys, mask, h * HU * VEC);
                }
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

// Called by every thread of a workgroup after its global atomics: true in the one
// workgroup that finishes last.  Values that cross workgroups go through
// device-wide read-modify-write atomics, which are coherent across the chip's L2
// caches: each thread waits until its own atomics are acknowledged before the
// barrier, so they precede the workgroup's increment of the counter, and the last
// workgroup reads them with read-modify-write atomics too.  (An agent-scope fence
// would write back and invalidate the L2 in every wave of every workgroup.)
__device__ __forceinline__ bool last_workgroup(uint32_t *done, uint32_t *flag) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t before = atomicAdd(done, 1u);
        *flag = before == gridDim.x - 1 ? 1u : 0u;
    }
    __syncthreads();
    return *flag != 0;
}

// Number of bits needed to write v (0 for 0).
__device__ __forceinline__ uint32_t bit_length(uint32_t v) { return v ? 32u - __clz(v) : 0u; }

// Scratch of a workgroup that resolves a pending digit or the sample's bracket.
struct ResolveLds {
    uint64_t tot[kDigitBins];
    uint64_t wave_tot[kHistWaves];
    uint64_t v[8];
    uint32_t d[4];
};

// The pass the state slot describes, with its pending digit chosen: the digit d of
// the pending histogram where the count of matching keys with digit > d is < k_rem
// <= that count plus total[d] is appended to the prefix.  Every workgroup of the
// kernel does the same from the same totals, which the previous kernel completed
// (plain loads suffice after the kernel boundary).
__device__ __forceinline__ Pass resolve(const PruneState *__restrict__ S,
                                        const unsigned long long *__restrict__ totals,
                                        int key_bits, ResolveLds &L) {
    Pass P;
    P.prefix = S->prefix;
    P.hi = S->hi < uint32_t(key_bits) ? S->hi : uint32_t(key_bits);
    P.base = S->base;
    P.cand = S->from_cand != 0;
    P.k_rem = S->k_rem;
    P.n_last = S->n_last;
    const uint32_t width = S->pend_width < P.hi ? S->pend_width : P.hi;
    if (width == 0) return P;                           // uniform
    const unsigned long long *t = totals + size_t(S->pend_buf % kTotalsBuffers) * kDigitBins;
    const int bins = 1 << width;
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) L.tot[b] = t[b];
    if (threadIdx.x == 0) {                             // if no digit qualifies
        L.v[0] = uint64_t(P.prefix) << width;
        L.v[1] = uint64_t(P.k_rem);
        L.v[2] = 0;
    }
    __syncthreads();
    // thread t owns the digits bins-1-2t and bins-2-2t (descending order)
    const int d0 = bins - 1 - 2 * int(threadIdx.x), d1 = d0 - 1;
    const uint64_t a = d0 >= 0 ? L.tot[d0] : 0, b = d1 >= 0 ? L.tot[d1] : 0;
    const uint64_t incl = block_inclusive_scan(a + b, L.wave_tot);
    const uint64_t excl = incl - a - b;
    const uint64_t k = uint64_t(P.k_rem);
    if (excl < k && k <= incl) {                        // exactly one thread
        const bool first = k <= excl + a;
        const uint32_t d = first ? uint32_t(d0) : uint32_t(d1);
        L.v[0] = (uint64_t(P.prefix) << width) | d;
        L.v[1] = k - (first ? excl : excl + a);
        L.v[2] = first ? a : b;
    }
    __syncthreads();
    P.prefix = uint32_t(L.v[0]);
    P.hi -= width;
    P.k_rem = int64_t(L.v[1]);
    P.n_last = L.v[2];
    return P;
}

// The split pass's bracket [dlo, dhi] of fine first digits (the top FB bits of the
// key) from the sample (n_s keys out of the matrix's total_keys, a fraction f): it
// holds the k-th largest key's digit up to six standard deviations of the sample
// count (a binomial) plus 8 keys: keys above dhi number at most f*k - margin in the
// sample, keys at or above dlo at least f*k + margin.  `single` unless the
// bracket's predicted candidates exceed cand_limit.  Every workgroup of the split
// pass computes it.  Thread t holds the sample's fine totals under the coarse
// digits (the top CB bits) c0 = 2^CB-1-2t and c1 = c0-1, f[0..R) for c1 and
// f[R..2R) for c0, loaded by the caller in one round trip; the coarse totals are
// their sums, and the threads that hold the two ends' coarse digits find the ends
// among their fine digits.  Results in L.d[0] (dlo), L.d[1] (dhi), L.d[2] (single).
template <int CB_BITS, int FB_BITS>
__device__ __forceinline__ void bracket(const uint32_t (&f)[2 << (FB_BITS - CB_BITS)],
                                        int64_t total_keys, int64_t k, uint64_t cand_limit,
                                        ResolveLds &L) {
    constexpr int CB = 1 << CB_BITS;
    constexpr int R = 1 << (FB_BITS - CB_BITS);         // fine digits per coarse digit
    constexpr uint32_t kTop = (1u << FB_BITS) - 1;
    static_assert(CB <= 2 * kHistThreads, "two coarse digits per thread");
    const int c0 = CB - 1 - 2 * int(threadIdx.x), c1 = c0 - 1;
    uint64_t a = 0, b = 0;                              // the coarse totals of c0, c1
#pragma unroll
    for (int j = 0; j < R; ++j) {
        b += f[j];
        a += f[R + j];
    }
    if (threadIdx.x == 0) {                             // an end no digit qualifies for
        L.d[0] = 0;                                     // dlo: the whole range
        L.d[1] = kTop;                                  // dhi: the whole range
        L.v[1] = 0;                                     // sample keys above dhi
    }
    const uint64_t incl = block_inclusive_scan(a + b, L.wave_tot);
    const uint64_t excl = incl - a - b;
    if (threadIdx.x == kHistThreads - 1) L.v[4] = incl;
    __syncthreads();
    const uint64_t n_s = L.v[4];
    if (threadIdx.x == 0) L.v[0] = n_s;                 // sample keys at or above dlo
    __syncthreads();
    const double q = double(k) / double(total_keys);
    const double ks = q * double(n_s);
    const double margin = 6.0 * sqrt(ks * (1.0 - q)) + 8.0;
    const double lo = ks - margin, hi = ks + margin;
    // digit d has `above` keys with a larger digit and `above + c` at or above it,
    // both non-increasing in d: dhi is the one digit with above <= lo < above + c
    // (or digit 0 with above <= lo), dlo the one with above < hi <= above + c (or
    // the top digit with above + c >= hi); first among the coarse digits, then among
    // the fine digits of the coarse digit found (its whole range if they disagree)
    auto ends = [&](int c, uint64_t above, uint64_t cnt, int fo) {
        if (c < 0) return;
        const double ab = double(above), at = double(above + cnt);
        if (ab <= lo && (c == 0 || at > lo)) {
            uint32_t dhi = uint32_t(c) * R + R - 1;
            uint64_t above_hi = above, x = above;
            for (int j = R - 1; j >= 0; --j) {
                const uint32_t fd = uint32_t(c) * R + uint32_t(j);
                if (double(x) <= lo && (fd == 0 || double(x + f[fo + j]) > lo)) {
                    dhi = fd;
                    above_hi = x;
                    break;
                }
                x += f[fo + j];
            }
            L.d[1] = dhi;
            L.v[1] = above_hi;
        }
        if (at >= hi && (c == CB - 1 || ab < hi)) {
            uint32_t dlo = uint32_t(c) * R;
            uint64_t at_lo = above + cnt, x = above;
            for (int j = R - 1; j >= 0; --j) {
                if (double(x + f[fo + j]) >= hi) {
                    dlo = uint32_t(c) * R + uint32_t(j);
                    at_lo = x + f[fo + j];
                    break;
                }
                x += f[fo + j];
            }
            L.d[0] = dlo;
            L.v[0] = at_lo;
        }
    };
    ends(c0, excl, a, R);
    ends(c1, excl + a, b, 0);
    __syncthreads();
    if (threadIdx.x == 0) {
        // predicted candidates: the bracket's sample keys scaled by 1/f
        const uint32_t dlo = L.d[0], dhi = L.d[1];
        const uint64_t at_lo = L.v[0], above_hi = L.v[1];
        const bool ok = dlo <= dhi && at_lo >= above_hi;
        const uint64_t in_all = ok ? at_lo - above_hi : 0;
        const bool fits = ok && n_s > 0 && double(in_all) * double(total_keys) <=
                                               double(cand_limit) * double(n_s);
        L.d[2] = fits ? 1u : 0u;
    }
    __syncthreads();
}

// What a histogram pass is for.
enum HistRole {
    kRoleNext = 0,        // the next digit, as the state describes it
    kRoleAfterSplit = 1,  // the first pass after the split: from the candidates if they
                          // hold the threshold, else from W (from the first digit on)
};

// The pass after a split pass that kept the sample's bracket: over the candidates'
// keys relative to the bracket's lowest key when G < k <= G + candidates (G the
// keys above the bracket), else over all of W from the first digit.  `cap` bounds
// the candidate count read back.
template <typename Bits>
__device__ __forceinline__ Pass pass_after_split(const SplitInfo *__restrict__ I, int64_t k,
                                                 uint64_t cap) {
    constexpr int KB = PruneTraits<Bits>::KEY_BITS;
    constexpr int first_shift = KB - PruneTraits<Bits>::SAMPLE_BITS;
    Pass P;
    const uint64_t G = I->n_above, n = I->n_cand, kk = uint64_t(k);
    const uint32_t dlo = I->dlo, dhi = I->dhi;
    P.prefix = 0;
    P.n_last = 0;
    if (!I->overflow && n <= cap && dlo <= dhi && G < kk && kk <= G + n) {
        P.base = dlo << first_shift;
        P.hi = uint32_t(first_shift) + bit_length(dhi - dlo);
        P.cand = true;
        P.k_rem = int64_t(kk - G);
    } else {
        P.base = 0;
        P.hi = KB;
        P.cand = false;
        P.k_rem = k;
    }
    return P;
}

// The pass before any digit is chosen: prefix 0, every key bit left, base 0, K to find.
__device__ __forceinline__ Pass first_pass(int key_bits, int64_t k) {
    Pass P;
    P.prefix = 0;
    P.hi = uint32_t(key_bits);
    P.base = 0;
    P.cand = false;
    P.k_rem = k;
    P.n_last = 0;
    return P;
}

// Write the state slot the next kernel reads: pass P, with its digit of `width`
// bits pending in totals buffer `buf` (width 0: nothing pending).
__device__ __forceinline__ void hand_on(PruneState *__restrict__ out, const Pass &P, int width,
                                        int buf) {
    out->prefix = P.prefix;
    out->hi = P.hi;
    out->base = P.base;
    out->from_cand = P.cand ? 1u : 0u;
    out->k_rem = P.k_rem;
    out->n_last = P.n_last;
    out->pend_width = uint32_t(width);
    out->pend_buf = uint32_t(buf);
}

// A histogram pass: the pending digit chosen, the next digit's histogram (over W or
// the candidates) into totals buffer `buf`.  Over candidates only the workgroups
// they fill take part, and their keys are loaded before the pending digit is
// chosen (one memory latency for both).  A pass that would find every bit chosen
// once the pending digit is leaves that digit to the count and hands the state on.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_hist_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave,
    PruneState *__restrict__ slots, const SplitInfo *__restrict__ info,
    unsigned long long *__restrict__ totals, const uint64_t *__restrict__ cand, int rd, int buf,
    int role, int64_t k, uint64_t cap) {
    constexpr int kStride = (1 << kMaxDigitBits) + 1;   // copies land in different banks
    constexpr int KB = PruneTraits<Bits>::KEY_BITS;
    __shared__ uint32_t hist[kCopies * kStride];
    __shared__ ResolveLds L;
    const PruneState *S = slots + rd;
    const bool derived = role == kRoleAfterSplit && info->single;   // uniform
    Pass P;
    bool from_cand;
    if (derived) {
        P = pass_after_split<Bits>(info, k, cap);
        from_cand = P.cand;
    } else {
        const uint32_t hi = S->hi < uint32_t(KB) ? S->hi : uint32_t(KB);
        if (hi <= S->pend_width) {                      // nothing after the pending digit
            if (blockIdx.x == 0 && threadIdx.x == 0) slots[rd ^ 1] = *S;
            return;
        }
        from_cand = S->from_cand != 0;
    }
    uint64_t n = 0;
    uint32_t active = gridDim.x;
    const uint64_t per_group = uint64_t(kCandPerThread) * kHistThreads;
    if (from_cand) {
        n = info->n_cand;
        if (n > cap) n = cap;
        // kCandPerThread candidates per thread: few workgroups, so few bins to flush
        const uint64_t g = n > per_group ? (n + per_group - 1) / per_group : 1;
        if (g < active) active = uint32_t(g);
    }
    if (blockIdx.x >= active) return;                   // uniform; workgroup 0 stays
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
    if (from_cand) load_batch();
    asm volatile("" ::: "memory");                      // the loads go out first
    if (!derived) P = resolve(S, totals, KB, L);
    const int width = digit_width(int(P.hi));
    if (blockIdx.x == 0 && threadIdx.x == 0) hand_on(slots + (rd ^ 1), P, width, buf);
    const int bins = 1 << width;
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
    if (from_cand) {
        // all of a batch's loads issued before its LDS atomics
        while (i0 < n) {
#pragma unroll
            for (int j = 0; j < kCandPerThread; ++j)
                if (i0 + uint64_t(j) * stride < n) add(kk[j]);
            i0 += stride * kCandPerThread;
            if (i0 < n) load_batch();
        }
    } else {
        for_each_key<Bits, ALIGNED>(W, ldw, M, N, per_wave, per_wave, [](int64_t) {}, add);
    }
    __syncthreads();
    unsigned long long *total = totals + size_t(buf) * kDigitBins;
    for (int b = int(threadIdx.x); b < bins; b += kHistThreads) {
        uint32_t v = 0;
#pragma unroll
        for (int c = 0; c < kCopies; ++c) v += hist[c * kStride + b];
        if (v) atomicAdd(&total[b], (unsigned long long)v);
    }
}

// The first kernel of a call that splits: the state reset (as prune_init_kernel,
// except `fine`, which the previous call's count left at zero), then the sample:
// the histogram of the keys' first SAMPLE_BITS bits over ranges of chunk elements
// range_stride apart (one range per wave), added into `fine` (32-bit totals: only
// the bracket depends on them, and a bracket that misses the K-th key, as one from
// a workspace that held something else would, costs passes over W, not exactness).
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_sample_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t chunk,
    int64_t range_stride, uint32_t *__restrict__ fine, int64_t k, PruneState *slots,
    SplitInfo *info, int64_t *counts, int64_t *eq, int64_t *gt1, uint64_t *totals) {
    constexpr int KB = PruneTraits<Bits>::KEY_BITS;
    constexpr int FB = PruneTraits<Bits>::SAMPLE_BITS;
    constexpr uint32_t shift = uint32_t(KB - FB);
    __shared__ uint32_t hist[1 << FB];
    for (int i = int(threadIdx.x); i < (1 << FB); i += kHistThreads) hist[i] = 0;
    {
        const int64_t stride = int64_t(gridDim.x) * kHistThreads;
        const int64_t first = int64_t(blockIdx.x) * kHistThreads + threadIdx.x;
        for (int64_t i = first; i < M; i += stride) {
            counts[i] = 0;
            eq[i] = 0;
            gt1[i] = 0;
        }
        for (int64_t i = first; i < int64_t(kTotalsBuffers) * kDigitBins; i += stride)
            totals[i] = 0;
        if (first == 0) {
            *info = SplitInfo{};
            hand_on(slots, first_pass(KB, k), 0, 0);
        }
    }
    __syncthreads();
    for_each_key<Bits, ALIGNED>(W, ldw, M, N, chunk, range_stride, [](int64_t) {},
                                [&](uint32_t key) { atomicAdd(&hist[key >> shift], 1u); });
    __syncthreads();
    for (int b = int(threadIdx.x); b < (1 << FB); b += kHistThreads) {
        const uint32_t v = hist[b];
        if (v) atomicAdd(&fine[b], v);
    }
}

// The split pass.  Every workgroup computes the sample's bracket [dlo, dhi] of fine
// first digits while the lines of its first round of W are on their way to the L2
// (the sample's totals are requested first).  With `single`, per row the keys
// with first digit > dhi go to gt1 (and their total to the split info's n_above)
// and the keys inside the bracket are stored as (row << 32 | key) candidates; if a
// wave's candidates overflow its LDS region or the workspace's room, the overflow
// flag sends the later passes back to W.  Without `single` (the bracket would hold
// too many keys) it takes the histogram of the first digit over W instead, into
// totals buffer `buf`.  Runs in the same grid as the histogram passes.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_split_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave,
    PruneState *__restrict__ slots, SplitInfo *__restrict__ info,
    unsigned long long *__restrict__ totals, const uint32_t *__restrict__ fine,
    unsigned long long *__restrict__ gt1, uint64_t *__restrict__ cand, uint64_t cap, int rd,
    int buf, int64_t k, uint64_t cand_limit) {
    constexpr int kStride = (1 << kMaxDigitBits) + 1;
    constexpr int KB = PruneTraits<Bits>::KEY_BITS;
    constexpr int FB = PruneTraits<Bits>::SAMPLE_BITS;
    constexpr int CB = digit_width(KB);
    constexpr int first_shift = KB - FB;
    constexpr uint32_t hist_shift = uint32_t(KB - CB);
    static_assert(kWaveRoom * kHistWaves == kSplitLds, "one LDS region per wave");
    __shared__ uint64_t buf_lds[kSplitLds];
    __shared__ uint32_t hist[kCopies * kStride];
    __shared__ ResolveLds L;
    __shared__ uint32_t wave_n[kHistWaves];
    __shared__ uint64_t base;
    // the sample's fine totals under this thread's two coarse digits
    // ((1<<CB)-2-2t and (1<<CB)-1-2t: 2R consecutive totals, 16-byte loads)
    constexpr int R = 1 << (FB - CB);
    static_assert((2 * R) % 4 == 0, "whole 16-byte loads");
    uint32_t ft[2 * R];
    {
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const int c1 = (1 << CB) - 2 - 2 * int(threadIdx.x);
        const u32x4 *src = reinterpret_cast<const u32x4 *>(fine + (c1 >= 0 ? c1 : 0) * R);
#pragma unroll
        for (int i = 0; i < 2 * R / 4; ++i) {
            const u32x4 v = src[i];
#pragma unroll
            for (int e = 0; e < 4; ++e) ft[4 * i + e] = c1 >= 0 ? v[e] : 0u;
        }
    }
    asm volatile("" ::: "memory");                      // these loads go out first
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
    uint64_t *mine = buf_lds + wave * kWaveRoom;
    uint32_t *hmine = hist + (int(threadIdx.x) & (kCopies - 1)) * kStride;
    uint32_t dlo = 0, dhi = 0;
    bool single = true;
    // the bracket, the split info and the next state slot (and, without `single`,
    // the cleared histogram)
    auto hook = [&]() {
        bracket<CB, FB>(ft, M * N, k, cand_limit, L);
        dlo = L.d[0];
        dhi = L.d[1];
        single = L.d[2] != 0;                           // uniform
        if (blockIdx.x == 0 && threadIdx.x == 0) {
            info->single = single ? 1u : 0u;
            info->dlo = dlo;
            info->dhi = dhi;
            // nothing chosen yet
            hand_on(slots + (rd ^ 1), first_pass(KB, k), single ? 0 : CB, buf);
        }
        if (!single) {
            for (int i = int(threadIdx.x); i < kCopies * kStride; i += kHistThreads) hist[i] = 0;
            __syncthreads();
        }
    };
    // the wave's candidates so far and its keys above the bracket (wave-uniform):
    // each wave fills its own LDS region, so no atomic sits between a round's keys
    // and the next round's loads
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
    {
        // request the lines of the wave's first round now (plain loads: they stay in
        // the L2), so that the bracket's two round trips overlap that round's
        // latency instead of preceding it
        constexpr int VEC = PruneTraits<Bits>::VEC;
        const int64_t Np = padded_n<Bits>(N);
        const int64_t a = (int64_t(blockIdx.x) * kHistWaves + wave) * per_wave;
        constexpr int U = PruneTraits<Bits>::UNROLL;
        // unconditional (a wave without a range reads row 0, indices are clamped into
        // the row): the compiler then waits for the older coarse totals alone
        const int64_t a0 = a < M * Np ? a : 0;
        const int64_t r = a0 / Np, c = a0 - r * Np;
        const Bits *row = W + r * ldw;
        uint32_t warm[U];
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const int64_t cc = c + int64_t(q) * kWave * VEC + int64_t(lane) * VEC;
            warm[q] = uint32_t(row[cc < N ? cc : N - 1]);
        }
        hook();
#pragma unroll
        for (int q = 0; q < U; ++q) asm volatile("" ::"v"(warm[q]));   // used (and done) here
    }
    auto on_unit = [&](int64_t r) {
        if (r != cur) {
            flush();
            cur = r;
        }
    };
    // the keys of a round (or of half a round), KN of them
    auto process = [&](const auto &keys, uint32_t mask) {
        constexpr int KN = int(std::extent<std::remove_reference_t<decltype(keys)>>::value);
        if (!single) {                                  // uniform: the first digit's histogram
#pragma unroll
            for (int j = 0; j < KN; ++j)
                if ((mask >> j) & 1u) atomicAdd(&hmine[keys[j] >> hist_shift], 1u);
            return;
        }
        // branch-free over the keys: the count above the bracket and a mask of the
        // candidates; then one ballot per key slot, and each lane places its own
        // candidates by the set bits below it in the ballot
        uint32_t cm = 0;
#pragma unroll
        for (int j = 0; j < KN; ++j) {
            const uint32_t top = keys[j] >> first_shift;
            const bool in = (mask >> j) & 1u;
            n_gt += (in && top > dhi) ? 1u : 0u;
            cm |= (in && top >= dlo && top <= dhi) ? (1u << j) : 0u;
        }
#pragma unroll
        for (int j = 0; j < KN; ++j) {
            const uint64_t bal = __ballot((cm >> j) & 1u);
            if (bal) {                                  // wave-uniform
                const uint32_t p = wn + __builtin_amdgcn_mbcnt_hi(
                                             uint32_t(bal >> 32),
                                             __builtin_amdgcn_mbcnt_lo(uint32_t(bal), 0u));
                if (((cm >> j) & 1u) && p < uint32_t(kWaveRoom))
                    mine[p] = (uint64_t(cur) << 32) | keys[j];
                wn += uint32_t(__popcll(bal));
            }
        }
    };
    if constexpr (ALIGNED) {
        constexpr int KH = K / 2;
        for_each_round_halves<Bits>(W, ldw, M, N, per_wave, on_unit,
                                    [&](const uint32_t (&keys)[KH], uint32_t mask, int) {
                                        process(keys, mask);
                                    });
    } else {
        for_each_round<Bits, false>(W, ldw, M, N, per_wave, per_wave, on_unit,
                                    [&](const uint32_t (&keys)[K], uint32_t mask) {
                                        process(keys, mask);
                                    });
    }
    if (!single) {                                      // uniform
        __syncthreads();
        unsigned long long *total = totals + size_t(buf) * kDigitBins;
        for (int b = int(threadIdx.x); b < (1 << CB); b += kHistThreads) {
            uint32_t v = 0;
#pragma unroll
            for (int c = 0; c < kCopies; ++c) v += hist[c * kStride + b];
            if (v) atomicAdd(&total[b], (unsigned long long)v);
        }
        return;
    }
    flush();
    if (lane == 0) {
        wave_n[wave] = wn;
        L.wave_tot[wave] = w_above;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t n = 0;
        bool over = false;
        uint64_t above = 0;
        for (int w = 0; w < kHistWaves; ++w) {
            n += wave_n[w];
            over = over || wave_n[w] > uint32_t(kWaveRoom);
            above += L.wave_tot[w];
        }
        uint64_t b = 0;
        if (over) {
            atomicExch(&info->overflow, 1u);
            b = cap;                                    // nothing is copied
        } else if (n > 0) {
            b = atomicAdd(&info->n_cand, (unsigned long long)n);
            if (b + n > cap) {
                atomicExch(&info->overflow, 1u);
                b = cap;
            }
        }
        if (above) atomicAdd(&info->n_above, (unsigned long long)above);
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
__device__ __forceinline__ void take_ties(int64_t M, int64_t need,
                                          unsigned long long *__restrict__ counts,
                                          unsigned long long *__restrict__ eq,
                                          uint64_t *wave_tot, int64_t *tile_total) {
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

// Per-row counts of keys > t (into counts) and == t (into eq); t = base + prefix
// once the pending digit is chosen.  From the candidates when they hold the
// threshold (plus the split pass's gt1), else from W.  When only some keys == t
// are kept, the last workgroup to finish then adds those.
template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kHistThreads) void prune_count_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t M, int64_t N, int64_t per_wave,
    const PruneState *__restrict__ slots, SplitInfo *__restrict__ info,
    const unsigned long long *__restrict__ totals, unsigned long long *__restrict__ gt,
    unsigned long long *__restrict__ eq, const uint64_t *__restrict__ cand,
    const unsigned long long *__restrict__ gt1, uint64_t cap, int rd,
    uint32_t *__restrict__ fine) {
    constexpr int KB = PruneTraits<Bits>::KEY_BITS;
    __shared__ ResolveLds L;
    __shared__ int64_t tile_total;
    __shared__ uint32_t flag;
    const int lane = int(threadIdx.x) & (kWave - 1);
    // over candidates, this lane's first one is loaded before the pending digit is
    // chosen (one memory latency for both)
    const bool from_cand = slots[rd].from_cand != 0;   // uniform
    uint64_t n = 0;
    if (from_cand) {
        n = info->n_cand;
        if (n > cap) n = cap;
    }
    const uint64_t stride = uint64_t(gridDim.x) * kHistThreads;
    const uint64_t first = uint64_t(blockIdx.x) * kHistThreads + threadIdx.x;
    uint64_t c_next = from_cand && first < n ? cand[first] : 0;
    asm volatile("" ::: "memory");                      // the load goes out first
    const Pass P = resolve(slots + rd, totals, KB, L);
    // the sample histogram is spent: zero it for the next call's sample
    for (uint64_t i = first; i < uint64_t(kFineBins); i += stride) fine[i] = 0;
    const uint32_t t = P.base + P.prefix;
    // when every key equal to t is taken (always, without ties), they count with the
    // keys above t and nothing is left for the last workgroup
    const bool all_ties = P.n_last == (unsigned long long)P.k_rem;
    unsigned long long *__restrict__ eqc = all_ties ? gt : eq;
    if (from_cand) {                                    // uniform
        // a wave's 64 candidates come in runs from few rows (each run is one
        // wave-round of the split pass): one atomic per row present and kind
        for (uint64_t i0 = first - uint64_t(lane); i0 < n; i0 += stride) {   // wave-uniform
            const uint64_t i = i0 + uint64_t(lane);
            const uint64_t c = c_next;
            c_next = i + stride < n ? cand[i + stride] : 0;
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
    if (last_workgroup(&info->done, &flag))
        take_ties(M, P.k_rem, gt, eq, L.wave_tot, &tile_total);
}

// Zero counts, eq, gt1, the split info and every totals buffer, and write state
// slot 0: nothing chosen yet (prefix 0, hi = the key's bits, base 0, k_rem = k).
__global__ __launch_bounds__(256) void prune_init_kernel(int64_t M, int64_t k, int key_bits,
                                                         PruneState *slots, SplitInfo *info,
                                                         int64_t *counts, int64_t *eq,
                                                         int64_t *gt1, uint64_t *totals,
                                                         uint32_t *fine) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i < M) {
        counts[i] = 0;
        eq[i] = 0;
        gt1[i] = 0;
    }
    if (i < int64_t(kTotalsBuffers) * kDigitBins) totals[i] = 0;
    if (i < kFineBins) fine[i] = 0;
    if (i == 0) {
        *info = SplitInfo{};
        hand_on(slots, first_pass(key_bits, k), 0, 0);
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

// Workspace: the two state slots and the split info, the totals buffers, the
// sample's fine totals, the per-row counts of keys equal to the threshold and of
// keys above the first digit, then the candidates.
struct PruneWorkspace {
    PruneState *slots;      // [2]
    SplitInfo *info;
    uint64_t *totals;       // [kTotalsBuffers][kDigitBins]
    uint32_t *fine;         // [kFineBins]
    int64_t *eq;            // [M]
    int64_t *gt1;           // [M]
    uint64_t *cand;         // [cand_capacity]
};

struct PruneOffsets { int64_t info, totals, fine, eq, gt1, cand, bytes; };

PruneOffsets prune_offsets(int64_t M, int64_t N) {
    PruneOffsets o;
    o.info = align256(2 * int64_t(sizeof(PruneState)));
    o.totals = o.info + align256(int64_t(sizeof(SplitInfo)));
    o.fine = o.totals + align256(int64_t(kTotalsBuffers) * kDigitBins * 8);
    o.eq = o.fine + align256(int64_t(kFineBins) * 4);
    o.gt1 = o.eq + align256(M * int64_t(sizeof(int64_t)));
    o.cand = o.gt1 + align256(M * int64_t(sizeof(int64_t)));
    o.bytes = o.cand + align256(cand_capacity(M, N) * int64_t(sizeof(uint64_t)));
    return o;
}

PruneWorkspace prune_workspace(int64_t M, int64_t N, void *base) {
    const PruneOffsets o = prune_offsets(M, N);
    char *c = static_cast<char *>(base);
    PruneWorkspace w;
    w.slots = reinterpret_cast<PruneState *>(c);
    w.info = reinterpret_cast<SplitInfo *>(c + o.info);
    w.totals = reinterpret_cast<uint64_t *>(c + o.totals);
    w.fine = reinterpret_cast<uint32_t *>(c + o.fine);
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
    auto *totals_u = reinterpret_cast<unsigned long long *>(w.totals);
    const PrunePartition part = prune_partition<Bits>(M, N);
    const int groups = part.groups;
    const int64_t per_wave = part.per_wave;
    constexpr int64_t kInitMin = int64_t(kTotalsBuffers) * kDigitBins > kFineBins
                                     ? int64_t(kTotalsBuffers) * kDigitBins
                                     : int64_t(kFineBins);
    const int64_t init_n = M > kInitMin ? M : kInitMin;
    const int64_t init_blocks = (init_n + 255) / 256;
    if (init_blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    // the state reset: its own launch, unless the sample (the first kernel of a call
    // that splits) does it
    const bool split = k > 0 && M * N * int64_t(sizeof(Bits)) >= kSplitMinBytes;
    if (!split)
        hipLaunchKernelGGL(prune_init_kernel, dim3(unsigned(init_blocks)), dim3(256), 0, s, M,
                           k, int(Tr::KEY_BITS), w.slots, w.info, counts, w.eq, w.gt1, w.totals,
                           w.fine);
    if (k == 0) return hipGetLastError();               // nothing kept: counts stay 0

    const bool aligned = (reinterpret_cast<uintptr_t>(W) % 16 == 0) &&
                         ((ldw * int64_t(sizeof(Bits))) % 16 == 0);
    // digits of the whole key (3 for fp32, 2 for fp16): every way through the
    // passes needs at most that many after the split
    constexpr int passes = digit_passes(Tr::KEY_BITS);
    static_assert(kBufPass0 + passes <= kTotalsBuffers, "a totals buffer per pass");
    const uint64_t cap = uint64_t(cand_room);
    auto *gt1_u = reinterpret_cast<unsigned long long *>(w.gt1);
    // more predicted candidates than this and the split pass takes the first digit
    const uint64_t cand_limit =
        std::min<uint64_t>(cap / 2, uint64_t(groups) * uint64_t(kSplitLds) / 2);
    int rd = 0;                                         // the state slot the next kernel reads
    auto hist = [&](int buf, int role) {
        if (aligned)
            hipLaunchKernelGGL((prune_hist_kernel<Bits, true>), dim3(groups), dim3(kHistThreads),
                               0, s, W, ldw, M, N, per_wave, w.slots, w.info, totals_u, w.cand,
                               rd, buf, role, k, cap);
        else
            hipLaunchKernelGGL((prune_hist_kernel<Bits, false>), dim3(groups),
                               dim3(kHistThreads), 0, s, W, ldw, M, N, per_wave, w.slots, w.info,
                               totals_u, w.cand, rd, buf, role, k, cap);
        rd ^= 1;
    };
    // the split pass pays for its extra launches only on large matrices: below
    // kSplitMinBytes of W every pass streams W
    if (split) {
        // the sample (ranges of kSampleChunk vectors per lane, one out of about every
        // kSampleEvery, the stride drifting by an odd number of vectors so that it
        // does not follow power-of-two rows), in as many workgroups as it has ranges
        // for; the split pass then reads W once
        const int64_t chunk = kSampleChunk * int64_t(kWave) * Tr::VEC;
        const int64_t range_stride = kSampleEvery * chunk + kSampleDrift * Tr::VEC;
        const int64_t ranges = (M * padded_n<Bits>(N) + range_stride - 1) / range_stride;
        const int64_t sample_groups =
            std::min<int64_t>(kSampleGroups, (ranges + kHistWaves - 1) / kHistWaves);
        const dim3 sgrid(unsigned(std::max<int64_t>(1, sample_groups)));
        if (aligned)
            hipLaunchKernelGGL((prune_sample_kernel<Bits, true>), sgrid, dim3(kHistThreads), 0, s,
                               W, ldw, M, N, chunk, range_stride, w.fine, k, w.slots, w.info,
                               counts, w.eq, w.gt1, w.totals);
        else
            hipLaunchKernelGGL((prune_sample_kernel<Bits, false>), sgrid, dim3(kHistThreads), 0,
                               s, W, ldw, M, N, chunk, range_stride, w.fine, k, w.slots, w.info,
                               counts, w.eq, w.gt1, w.totals);
        if (aligned)
            hipLaunchKernelGGL((prune_split_kernel<Bits, true>), dim3(groups), dim3(kHistThreads),
                               0, s, W, ldw, M, N, per_wave, w.slots, w.info, totals_u, w.fine,
                               gt1_u, w.cand, cap, rd, kBufSplit, k, cand_limit);
        else
            hipLaunchKernelGGL((prune_split_kernel<Bits, false>), dim3(groups),
                               dim3(kHistThreads), 0, s, W, ldw, M, N, per_wave, w.slots, w.info,
                               totals_u, w.fine, gt1_u, w.cand, cap, rd, kBufSplit, k,
                               cand_limit);
        rd ^= 1;
        for (int p = 0; p < passes; ++p) hist(kBufPass0 + p, p == 0 ? kRoleAfterSplit : kRoleNext);
    } else {
        for (int p = 0; p < passes; ++p) hist(kBufPass0 + p, kRoleNext);
    }
    auto *gt_u = reinterpret_cast<unsigned long long *>(counts);
    auto *eq_u = reinterpret_cast<unsigned long long *>(w.eq);
    if (aligned)
        hipLaunchKernelGGL((prune_count_kernel<Bits, true>), dim3(groups), dim3(kHistThreads), 0,
                           s, W, ldw, M, N, per_wave, w.slots, w.info, totals_u, gt_u, eq_u,
                           w.cand, gt1_u, cap, rd, w.fine);
    else
        hipLaunchKernelGGL((prune_count_kernel<Bits, false>), dim3(groups), dim3(kHistThreads), 0,
                           s, W, ldw, M, N, per_wave, w.slots, w.info, totals_u, gt_u, eq_u,
                           w.cand, gt1_u, cap, rd, w.fine);
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
