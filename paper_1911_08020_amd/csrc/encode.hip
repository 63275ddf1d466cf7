// BMWM encode on gfx950 (section 3.1 block-max weight masking, with the
// per-row block size of section 3.2).
//
// Work unit: one wavefront handles one chunk of CHUNK consecutive columns of one
// row.  CHUNK is a multiple of every block size (<= 128), so no block straddles
// two waves.  Each lane loads VEC consecutive elements per 16-byte load, UNROLL
// loads in flight per lane, all issued before any compare (the kernel is bound
// by the HBM stream of the dense W).
//
// Selection: the magnitude key of an element is its bit pattern with the sign
// cleared.  Within a lane the VEC elements are scanned in column order with a
// strict ">" (earliest wins ties).  A block wider than VEC spans b/VEC
// consecutive lanes; their candidates are packed as
//     (magnitude << 8) | ((127 - j) << 1) | sign,     j = column within the block,
// so one unsigned max over an xor butterfly picks the largest magnitude and,
// among equal magnitudes, the smallest j; the sign travels along to rebuild the
// value.  Columns past N (tail block) load as +0.0 with their own j, so they can
// never beat a real column of the same block.  The butterfly's lane exchanges are
// DPP / swizzle register moves chosen at compile time per block size.
#include <type_traits>

#include "darb_internal.h"

namespace darb {
namespace {

constexpr int kEncodeThreads = 256;
constexpr int kEncodeWaves = kEncodeThreads / kWave;

template <typename Bits> struct EncodeTraits;
template <> struct EncodeTraits<uint32_t> {
    static constexpr int VEC = 4;          // 16 bytes
    static constexpr int UNROLL = 4;       // 64 B in flight per lane
    static constexpr uint32_t MAG = 0x7FFFFFFFu;
    static constexpr int SIGN_SHIFT = 31;
    using Key = uint64_t;
};
template <> struct EncodeTraits<uint16_t> {
    static constexpr int VEC = 8;          // 16 bytes
    static constexpr int UNROLL = 4;
    static constexpr uint32_t MAG = 0x7FFFu;
    static constexpr int SIGN_SHIFT = 15;
    using Key = uint32_t;
};

template <typename Bits>
__device__ __forceinline__ typename EncodeTraits<Bits>::Key pack_key(Bits v, int j) {
    using Tr = EncodeTraits<Bits>;
    using Key = typename Tr::Key;
    const uint32_t mag = uint32_t(v) & Tr::MAG;
    const uint32_t sgn = uint32_t(v) >> Tr::SIGN_SHIFT;
    return (Key(mag) << 8) | Key((127 - j) << 1) | Key(sgn);
}

template <typename Bits>
__device__ __forceinline__ void unpack_key(typename EncodeTraits<Bits>::Key k, Bits &v, int &j) {
    using Tr = EncodeTraits<Bits>;
    const uint32_t mag = uint32_t(k >> 8);
    const uint32_t sgn = uint32_t(k) & 1u;
    v = Bits(mag | (sgn << Tr::SIGN_SHIFT));
    j = 127 - int((uint32_t(k) >> 1) & 127u);
}

// Partner exchange of a max-butterfly that merges the two halves (M lanes each) of
// every aligned group of 2M lanes.  Any pairing across the two halves works for a
// max-reduction: quad_perm swaps for M = 1, 2, the 8- and 16-lane mirrors for
// M = 4, 8 (all DPP, plain VALU), a swizzle swapping 16-lane halves for M = 16.
template <int M> __device__ __forceinline__ uint32_t xchg(uint32_t v) {
    if constexpr (M == 1) {
        return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0xB1, 0xF, 0xF, false));
    } else if constexpr (M == 2) {
        return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x4E, 0xF, 0xF, false));
    } else if constexpr (M == 4) {
        return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x141, 0xF, 0xF, false));
    } else if constexpr (M == 8) {
        return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x140, 0xF, 0xF, false));
    } else {
        static_assert(M == 16, "blocks span at most 32 lanes");
        return uint32_t(__builtin_amdgcn_ds_swizzle(int(v), (0x10 << 10) | 0x1F));
    }
}
template <int M> __device__ __forceinline__ uint64_t xchg_key(uint64_t k) {
    return (uint64_t(xchg<M>(uint32_t(k >> 32))) << 32) | xchg<M>(uint32_t(k));
}
template <int M> __device__ __forceinline__ uint32_t xchg_key(uint32_t k) { return xchg<M>(k); }

template <typename Bits, int VEC> struct alignas(16) Vec { Bits e[VEC]; };

// Blocks of b = 2^LB <= VEC elements: the lane's vector holds VEC / b whole blocks.
template <typename Bits, int VEC, int LB>
__device__ __forceinline__ void small_blocks(const Vec<Bits, VEC> &v, int64_t c0, int64_t nblk,
                                             Bits *__restrict__ values,
                                             uint8_t *__restrict__ offsets) {
    using Tr = EncodeTraits<Bits>;
    constexpr int b = 1 << LB;
    if constexpr (b <= VEC) {
#pragma unroll
        for (int s = 0; s < VEC; s += b) {
            const int64_t k = (c0 + s) >> LB;
            Bits best_bits = v.e[s];
            uint32_t best_mag = uint32_t(v.e[s]) & Tr::MAG;
            int best = 0;
#pragma unroll
            for (int j = 1; j < b; ++j) {
                const uint32_t mag = uint32_t(v.e[s + j]) & Tr::MAG;
                const bool take = mag > best_mag;
                best_mag = take ? mag : best_mag;
                best_bits = take ? v.e[s + j] : best_bits;
                best = take ? j : best;
            }
            if (k < nblk) {
                values[k] = best_bits;
                offsets[k] = uint8_t(best);
            }
        }
    }
}

// Blocks wider than VEC: each lane's candidate, then an xor butterfly over the
// b / VEC consecutive lanes that hold the block.  The UNROLL vectors of a lane are
// independent, so every butterfly step shuffles all of them at once and their
// latencies overlap.
template <typename Bits, int VEC, int UNROLL, int LB>
__device__ __forceinline__ void wide_blocks(const Vec<Bits, VEC> (&v)[UNROLL], int64_t cbase,
                                            int lane, int64_t nblk, Bits *__restrict__ values,
                                            uint8_t *__restrict__ offsets) {
    using Tr = EncodeTraits<Bits>;
    using Key = typename Tr::Key;
    constexpr int b = 1 << LB;
    constexpr int group = b / VEC;                     // 2 .. 32 lanes hold one block
    if constexpr (group >= 2) {
        Key key[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int64_t c0 = cbase + int64_t(u) * (kWave * VEC) + int64_t(lane) * VEC;
            Bits best_bits = v[u].e[0];
            uint32_t best_mag = uint32_t(v[u].e[0]) & Tr::MAG;
            int best = 0;
#pragma unroll
            for (int e = 1; e < VEC; ++e) {
                const uint32_t mag = uint32_t(v[u].e[e]) & Tr::MAG;
                const bool take = mag > best_mag;
                best_mag = take ? mag : best_mag;
                best_bits = take ? v[u].e[e] : best_bits;
                best = take ? e : best;
            }
            key[u] = pack_key<Bits>(best_bits, int(c0 & (b - 1)) + best);
        }
        auto step = [&](auto mc) {
            constexpr int M = decltype(mc)::value;
            if constexpr (M < group) {
#pragma unroll
                for (int u = 0; u < UNROLL; ++u) {
                    const Key other = xchg_key<M>(key[u]);
                    key[u] = other > key[u] ? other : key[u];
                }
            }
        };
        step(std::integral_constant<int, 1>{});
        step(std::integral_constant<int, 2>{});
        step(std::integral_constant<int, 4>{});
        step(std::integral_constant<int, 8>{});
        step(std::integral_constant<int, 16>{});
        if ((lane & (group - 1)) == 0) {
#pragma unroll
            for (int u = 0; u < UNROLL; ++u) {
                const int64_t k = (cbase + int64_t(u) * (kWave * VEC) + int64_t(lane) * VEC) >> LB;
                if (k < nblk) {
                    Bits val;
                    int j;
                    unpack_key<Bits>(key[u], val, j);
                    values[k] = val;
                    offsets[k] = uint8_t(j);
                }
            }
        }
    }
}

// Blocks of b <= VEC for all UNROLL vectors of the lane.
template <typename Bits, int VEC, int UNROLL, int LB>
__device__ __forceinline__ void small_blocks_all(const Vec<Bits, VEC> (&v)[UNROLL], int64_t cbase,
                                                 int lane, int64_t nblk,
                                                 Bits *__restrict__ values,
                                                 uint8_t *__restrict__ offsets) {
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
        small_blocks<Bits, VEC, LB>(v[u], cbase + int64_t(u) * (kWave * VEC) + int64_t(lane) * VEC,
                                    nblk, values, offsets);
}

template <typename Bits, bool ALIGNED>
__global__ __launch_bounds__(kEncodeThreads) void encode_kernel(
    const Bits *__restrict__ W, int64_t ldw, int64_t N, const int64_t *__restrict__ rowinfo,
    int64_t chunks_per_row, int cgroups, Bits *__restrict__ values,
    uint8_t *__restrict__ offsets) {
    using Tr = EncodeTraits<Bits>;
    constexpr int VEC = Tr::VEC;
    constexpr int UNROLL = Tr::UNROLL;
    constexpr int64_t CHUNK = int64_t(kWave) * VEC * UNROLL;

    // workgroup -> (original row r, group of kEncodeWaves chunks); all uniform.  The
    // W loads depend on nothing but r, so they issue first; the row's block size and
    // first output slot arrive from the per-row table while they are in flight.
    const int r = int(blockIdx.x) / cgroups;
    const int cg = int(blockIdx.x) - r * cgroups;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int64_t q = int64_t(cg) * kEncodeWaves + wave;
    if (q >= chunks_per_row) return;                  // wave-uniform, no barrier below
    const Bits *row = W + int64_t(r) * ldw;
    const int64_t info = rowinfo[r];

    // issue every load of this lane first
    Vec<Bits, VEC> v[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
        const int64_t c0 = q * CHUNK + int64_t(u) * (kWave * VEC) + int64_t(lane) * VEC;
        if (ALIGNED && c0 + VEC <= N) {
            typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
            const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(row + c0));
            v[u] = __builtin_bit_cast(Vec<Bits, VEC>, t);
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) v[u].e[e] = (c0 + e < N) ? row[c0 + e] : Bits(0);
        }
    }

    const int lb = int(info & 0xFF);
    const int64_t nblk = (N + (int64_t(1) << lb) - 1) >> lb;
    const int64_t out0 = info >> 8;
    const int64_t cbase = q * CHUNK;
    Bits *vo = values + out0;
    uint8_t *oo = offsets + out0;
    // one wave-uniform branch on the block size, straight-line code inside
    constexpr int LV = VEC == 4 ? 2 : 3;   // log2 VEC: blocks up to VEC stay inside a lane
    switch (lb) {
        case 0: small_blocks_all<Bits, VEC, UNROLL, 0>(v, cbase, lane, nblk, vo, oo); break;
        case 1: small_blocks_all<Bits, VEC, UNROLL, 1>(v, cbase, lane, nblk, vo, oo); break;
        case 2: small_blocks_all<Bits, VEC, UNROLL, 2>(v, cbase, lane, nblk, vo, oo); break;
        case 3:
            if constexpr (LV >= 3) small_blocks_all<Bits, VEC, UNROLL, 3>(v, cbase, lane, nblk, vo, oo);
            else wide_blocks<Bits, VEC, UNROLL, 3>(v, cbase, lane, nblk, vo, oo);
            break;
        case 4: wide_blocks<Bits, VEC, UNROLL, 4>(v, cbase, lane, nblk, vo, oo); break;
        case 5: wide_blocks<Bits, VEC, UNROLL, 5>(v, cbase, lane, nblk, vo, oo); break;
        case 6: wide_blocks<Bits, VEC, UNROLL, 6>(v, cbase, lane, nblk, vo, oo); break;
        default: wide_blocks<Bits, VEC, UNROLL, 7>(v, cbase, lane, nblk, vo, oo); break;
    }
}

template <typename Bits>
hipError_t launch_encode_t(const darb_plan &p, const void *W, int64_t ldw, void *values,
                           uint8_t *offsets, hipStream_t s) {
    using Tr = EncodeTraits<Bits>;
    constexpr int64_t CHUNK = int64_t(kWave) * Tr::VEC * Tr::UNROLL;
    const int64_t chunks = (p.N + CHUNK - 1) / CHUNK;
    const int64_t cgroups = (chunks + kEncodeWaves - 1) / kEncodeWaves;
    const int64_t blocks = p.M * cgroups;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const bool aligned = (reinterpret_cast<uintptr_t>(W) % 16 == 0) &&
                         ((ldw * int64_t(sizeof(Bits))) % 16 == 0);
    const Bits *w = static_cast<const Bits *>(W);
    Bits *vals = static_cast<Bits *>(values);
    if (aligned)
        hipLaunchKernelGGL((encode_kernel<Bits, true>), dim3(unsigned(blocks)),
                           dim3(kEncodeThreads), 0, s, w, ldw, p.N, p.d_rowinfo, chunks,
                           int(cgroups), vals, offsets);
    else
        hipLaunchKernelGGL((encode_kernel<Bits, false>), dim3(unsigned(blocks)),
                           dim3(kEncodeThreads), 0, s, w, ldw, p.N, p.d_rowinfo, chunks,
                           int(cgroups), vals, offsets);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_encode(const darb_plan &p, int wdtype, const void *W, int64_t ldw,
                         void *values, uint8_t *offsets, hipStream_t s) {
    if (wdtype == DARB_F32) return launch_encode_t<uint32_t>(p, W, ldw, values, offsets, s);
    return launch_encode_t<uint16_t>(p, W, ldw, values, offsets, s);
}

}  // namespace darb
