// DARB products on gfx950: y = W_darb x (SpMV) and Y = W_darb X (SpMM) -- the
// kernels and their launch templates, instantiated by product.hip (fp32 and fp16
// weights) and product_i8.hip (INT8 weights).
//
// Only retained weights are read (section 2), and each retained weight's
// in-block offset selects the one activation it multiplies (section 3.2):
//     y[r] = sum_k v[r,k] * x[k * b_r + off[r,k]].
// The grouped layout makes every block-size group a dense [rows x nblk] array.
// Every workgroup works inside one group, so the group's geometry is uniform:
// it is read with scalar loads, and the per-lane work starts with the loads that
// matter.  Loads are never placed under per-lane branches: addresses are clamped
// into the buffer and the unused lanes' results are masked, so a wave issues all
// of its loads back to back.
//
// SpMV: `lanes` lanes per row, 64 / lanes rows per wave; each lane holds up to
// kVmax 16-byte vectors of values (plus their offset bytes) in registers.  Every
// wave first issues its share of the loads that stage x into LDS, then the loads of
// its vectors, so both memory latencies overlap; the gathers then hit LDS.  (Gathers
// from L2 instead cost several times the staging, and the fp32 products keep the
// exact x.)  A row's partial sums are combined by a
// fixed-order lane reduction (DPP within 16-lane rows, then lane exchanges; the
// result is deterministic) and written in original row order.
//
// SpMM: lanes map to batch columns (X is [N x B] row-major, so one weight's
// activations X[c, :] are contiguous), CPL columns per lane with 16-byte loads, or
// narrower ones for small batches so that a row still spreads over up to 16 lanes
// and the launch over many waves.  Each wave loads its rows' (value, column)
// pairs with coalesced loads and broadcasts them across a row's lanes register to
// register (DPP, swizzle or readlane), gathering X rows kSpmmBatch at a time; the
// next round's pairs load while this round gathers.  Up to 8 waves split a row group's weights
// and their partial sums meet in LDS in a fixed order.
//
// Both products read the offsets either as one byte per retained weight or in the
// bit-packed form of section 4.2 (log2 b bits each, packed_bits.h); the two forms
// share every other step, so their results are bitwise identical.
#pragma once
#include <hip/hip_fp16.h>

#include <type_traits>
#include <utility>

#include "darb_internal.h"
#include "packed_bits.h"

namespace darb {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<__half>(__half v) { return __half2float(v); }
template <> __device__ __forceinline__ float to_f32<int8_t>(int8_t v) { return float(v); }

// INT8 weights carry one fp32 scale per row, applied once to the row's sum.
template <typename Tw> constexpr bool kScaled = std::is_same<Tw, int8_t>::value;

__device__ __forceinline__ float half_bits_to_f32(uint32_t h) {
    return __half2float(__ushort_as_half(uint16_t(h & 0xFFFFu)));
}

__device__ __forceinline__ int wave_uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// v plus its value in the lane DPP control CTRL selects (all rows and banks)
template <int CTRL> __device__ __forceinline__ float add_dpp(float v) {
    return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                   0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// v plus the value DPP control CTRL selects, in the 16-lane rows ROWS enables (other
// rows add +0.0, which leaves them unchanged)
template <int CTRL, int ROWS> __device__ __forceinline__ float add_dpp_rows(float v) {
    return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                   0, __builtin_bit_cast(int, v), CTRL, ROWS, 0xF, false));
}

// Sum over aligned groups of 2^lgL lanes (lgL <= 6, wave-uniform); the group's sum
// ends in its last lane.  The pairs are lanes 1 apart, then 2 (quad permutations),
// then mirrored inside 8 and 16 lanes (row_half_mirror, row_mirror): after these
// every lane of a 16-lane row holds the row's sum.  Rows then meet by broadcasts:
// row 1 adds row 0 and row 3 adds row 2 (row_bcast:15), then row 3 adds row 1
// (row_bcast:31).  Each step adds two partial sums of equal size, so the result
// depends only on lgL, and no step goes through LDS.
__device__ __forceinline__ float group_sum(float v, int lgL) {
    if (lgL >= 1) v = add_dpp<0xB1>(v);     // quad_perm [1, 0, 3, 2]
    if (lgL >= 2) v = add_dpp<0x4E>(v);     // quad_perm [2, 3, 0, 1]
    if (lgL >= 3) v = add_dpp<0x141>(v);    // row_half_mirror
    if (lgL >= 4) v = add_dpp<0x140>(v);    // row_mirror
    if (lgL >= 5) v = add_dpp_rows<0x142, 0xA>(v);   // row_bcast:15 into rows 1 and 3
    if (lgL >= 6) v = add_dpp_rows<0x143, 0x8>(v);   // row_bcast:31 into row 3
    return v;
}

// Uniform selection of a per-group table entry (compile-time indices only, so the
// table stays in scalar registers).
template <typename T>
__device__ __forceinline__ T pick(const T (&a)[kMaxBins], int g) {
    T r = a[0];
#pragma unroll
    for (int b = 1; b < kMaxBins; ++b) r = (b == g) ? a[b] : r;
    return r;
}

// The block-size group that workgroup `tile` of a launch belongs to.
__device__ __forceinline__ int block_group(const ProductSchedule &s, int tile) {
    int g = 0;
#pragma unroll
    for (int b = 1; b < kMaxBins; ++b)
        if (b < s.nbins && tile >= s.block_begin[b]) g = b;
    return g;
}

__device__ __forceinline__ int block_begin_of(const ProductSchedule &s, int g) {
    int r = s.block_begin[0];
#pragma unroll
    for (int b = 1; b < kMaxBins; ++b) r = (b == g) ? s.block_begin[b] : r;
    return r;
}

// ---------------------------------------------------------------------------------
// Offset sources.  A lane loads the indices of NV consecutive retained weights of a
// group (group slots j .. j + NV - 1, j a multiple of NV) as `Raw`, keeps them in
// registers while other loads are in flight, turns them into `Bits` when it needs
// them and reads index q with field().
// ---------------------------------------------------------------------------------

struct GroupOffsets {
    const uint8_t *u8;     // byte form: the group's first slot
    PackedGroup pk;        // packed form
};

__device__ __forceinline__ GroupOffsets group_offsets(const void *offs, const BinTable &bins,
                                                      int g) {
    GroupOffsets go;
    go.u8 = static_cast<const uint8_t *>(offs) + pick(bins.first_elem, g);
    go.pk = packed_group(static_cast<const uint32_t *>(offs), pick(bins.first_word, g),
                         pick(bins.log2b, g));
    return go;
}

template <int NV> struct U8Vec;
template <> struct U8Vec<1> { using T = uint8_t; };
template <> struct U8Vec<2> { using T = uint16_t; };
template <> struct U8Vec<4> { using T = uint32_t; };
template <> struct U8Vec<8> { using T = u32x2; };
template <> struct U8Vec<16> { using T = u32x4; };

template <bool PK, int NV> struct Off;

// one byte per weight: one NV-byte load (the caller guarantees its alignment)
template <int NV> struct Off<false, NV> {
    using Raw = typename U8Vec<NV>::T;
    using Bits = Raw;
    __device__ static Raw load(const GroupOffsets &go, int64_t j) {
        return *reinterpret_cast<const Raw *>(go.u8 + j);
    }
    __device__ static Bits bits(const Raw &r, const GroupOffsets &) { return r; }
    __device__ static int field(const Bits &b, int q, const GroupOffsets &) {
        if constexpr (NV <= 4) return int((uint32_t(b) >> (8 * q)) & 0xFFu);
        else return int((b[q >> 2] >> (8 * (q & 3))) & 0xFFu);
    }
    // the same with q a compile-time index (the block size is implied by the byte)
    template <int LB> __device__ static int field_c(const Bits &b, int q) {
        return field(b, q, GroupOffsets{});
    }
};

// packed, up to 4 indices (<= 28 bits): two words
template <int NV> struct Off<true, NV> {
    static_assert(NV <= 4, "wider vectors have their own specialisations");
    using Raw = PackedWords2;
    using Bits = uint32_t;
    __device__ static Raw load(const GroupOffsets &go, int64_t j) { return packed_load2(go.pk, j); }
    __device__ static Bits bits(const Raw &r, const GroupOffsets &) { return packed_bits32(r); }
    __device__ static int field(Bits b, int q, const GroupOffsets &go) {
        return packed_field(b, q, go.pk);
    }
    template <int LB> __device__ static int field_c(Bits b, int q) {
        return int((b >> (q * LB)) & ((1u << LB) - 1u));
    }
};

// packed, 8 indices (<= 56 bits): three words
template <> struct Off<true, 8> {
    using Raw = PackedWords3;
    using Bits = uint64_t;
    __device__ static Raw load(const GroupOffsets &go, int64_t j) { return packed_load3(go.pk, j); }
    __device__ static Bits bits(const Raw &r, const GroupOffsets &) { return packed_bits64(r); }
    __device__ static int field(Bits b, int q, const GroupOffsets &go) {
        return packed_field(b, q, go.pk);
    }
    template <int LB> __device__ static int field_c(Bits b, int q) {
        return int(uint32_t(b >> (q * LB)) & ((1u << LB) - 1u));
    }
};

// packed, 16 indices: two 8-index windows (j is a multiple of 16, so both lie in
// one run)
template <> struct Off<true, 16> {
    struct Raw { PackedWords3 lo, hi; };
    struct Bits { uint64_t lo, hi; };
    __device__ static Raw load(const GroupOffsets &go, int64_t j) {
        return Raw{packed_load3(go.pk, j), packed_load3(go.pk, j + 8)};
    }
    __device__ static Bits bits(const Raw &r, const GroupOffsets &) {
        return Bits{packed_bits64(r.lo), packed_bits64(r.hi)};
    }
    __device__ static int field(const Bits &b, int q, const GroupOffsets &go) {
        return q < 8 ? packed_field(b.lo, q, go.pk) : packed_field(b.hi, q - 8, go.pk);
    }
};

// ---------------------------------------------------------------------------------
// SpMV
// ---------------------------------------------------------------------------------

constexpr int kSpmvThreads = 256;
constexpr int kSpmvWaves = kSpmvThreads / kWave;
constexpr int kVmax = 8;                         // vectors per lane per round
constexpr int kLoopVmax = 4;                     // per round, in the looping general form
constexpr int kLdsMaxFloats = 16384;             // x staged in LDS up to 64 KiB
constexpr int64_t kLdsPerCu = 160 * 1024;        // LDS of one gfx950 CU

template <typename Tw> struct WVec;
template <> struct WVec<float> {
    static constexpr int VEC = 4;
    using V = f32x4;        // 4 values, 16 bytes
    __device__ static float get(const V &v, int i) { return v[i]; }
};
template <> struct WVec<__half> {
    static constexpr int VEC = 8;
    using V = u32x4;        // 8 fp16 values, 16 bytes
    __device__ static float get(const V &v, int i) {
        const uint32_t w = v[i >> 1];
        return half_bits_to_f32((i & 1) ? (w >> 16) : w);
    }
};
template <> struct WVec<int8_t> {
    static constexpr int VEC = 8;
    using V = u32x2;        // 8 INT8 codes, 8 bytes (with their 8 offset bytes: 16)
    __device__ static float get(const V &v, int i) {
        // sign-extend byte i & 3 of word i >> 2
        return float(int32_t(v[i >> 2] << (24 - 8 * (i & 3))) >> 24);
    }
};

// x (N elements) into LDS as fp32 through registers, in two halves so that other
// loads can be issued between them: issue() loads up to SB 16-byte vectors per
// thread (addresses clamped), commit() waits for them, widens and stores them, and
// copies the scalar tail.  The launcher picks SB so that one round covers x.
template <typename Tx, int SB> struct XStage {
    static constexpr int E = 16 / int(sizeof(Tx));
    u32x4 t[SB];
    int nv;
    __device__ __forceinline__ void issue(const Tx *__restrict__ x, int N) {
        const bool aligned = (reinterpret_cast<uintptr_t>(x) & 15) == 0;
        nv = aligned ? N / E : 0;
        const u32x4 *x4 = reinterpret_cast<const u32x4 *>(x);
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            if (u * kSpmvThreads < nv) {                  // wave-uniform: skip empty rounds
                const int i = u * kSpmvThreads + int(threadIdx.x);
                t[u] = x4[i < nv ? i : nv - 1];
            }
        }
    }
    __device__ __forceinline__ void commit(float *xs, const Tx *__restrict__ x, int N) const {
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            const int i = u * kSpmvThreads + int(threadIdx.x);
            if (i < nv) {
                if constexpr (sizeof(Tx) == 4) {
                    *reinterpret_cast<u32x4 *>(xs + i * E) = t[u];
                } else {
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        xs[i * E + 2 * h] = half_bits_to_f32(t[u][h]);
                        xs[i * E + 2 * h + 1] = half_bits_to_f32(t[u][h] >> 16);
                    }
                }
            }
        }
        for (int c = nv * E + int(threadIdx.x); c < N; c += kSpmvThreads)
            xs[c] = to_f32<Tx>(x[c]);
    }
};

// fp32 x straight into LDS: each wave moves 1 KiB chunks with direct global-to-LDS
// loads (lane i's 16 bytes land at chunk + 16 i), so no registers hold x on the way.
// stage_x_direct issues them; stage_x_tail copies the rest (a partial chunk)
// through registers.  The caller waits for the loads and synchronises the workgroup.
__device__ __forceinline__ void stage_x_direct(float *xs, const float *__restrict__ x, int N) {
    typedef __attribute__((address_space(1))) const float *gptr;
    typedef __attribute__((address_space(3))) void *lptr;
    const int wave = wave_uniform(int(threadIdx.x) / kWave);
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int chunks = N / (kWave * 4);
    for (int j = wave; j < chunks; j += kSpmvWaves)
        __builtin_amdgcn_global_load_lds((gptr)(x + (j * kWave + lane) * 4),
                                         (lptr)(xs + j * kWave * 4), 16, 0, 0);
}
__device__ __forceinline__ void stage_x_tail(float *xs, const float *__restrict__ x, int N) {
    for (int c = N / (kWave * 4) * (kWave * 4) + int(threadIdx.x); c < N; c += kSpmvThreads)
        xs[c] = x[c];
}

template <typename Tw, typename Tx, bool LDS, int SB, bool PK, bool LOOP>
__global__ __launch_bounds__(kSpmvThreads) void spmv_kernel(
    const Tw *__restrict__ values, const void *__restrict__ offs,
    const Tx *__restrict__ x, float *__restrict__ y, const int32_t *__restrict__ perm,
    int N, BinTable bins, ProductSchedule sch, const float *__restrict__ scales,
    int total_blocks) {
    using WV = WVec<Tw>;
    constexpr int VEC = WV::VEC;
    using OV = Off<PK, VEC>;
    using OS = Off<PK, 1>;
    // vectors per lane and round: the looping form keeps two blocks in registers, so it
    // holds half as many per round (its lanes take further rounds of vectors in the
    // same order: the lanes per row, and so the sums, are the one-pass form's)
    constexpr int KV = LOOP ? kLoopVmax : kVmax;
    extern __shared__ float xs[];

    const int wave = wave_uniform(int(threadIdx.x) / kWave);
    const int lane = int(threadIdx.x) & (kWave - 1);

    // A workgroup stages x once and then takes blocks blockIdx.x, + gridDim.x, ...
    // (LOOP; otherwise the grid has one workgroup per block and keeps one block's
    // state, so it needs fewer registers); each block is kSpmvWaves tiles of one
    // group.  A Tile holds one block's state: geometry() reads the block's group
    // geometry and issues the load of the lane's output row, issue() the first round of
    // the lane's vectors, finish() sums them and writes the row.  LOOP keeps two Tiles
    // and issues the next block's loads before summing the current one.
    struct Tile {
        int g, lgL, L, lb, nblk, sub, nvec;
        int64_t j0, e0;
        bool vec_path, whole, row_ok;
        GroupOffsets go;
        int32_t dest;
        float scale;
        const typename WV::V *vrow;
        typename WV::V wv[KV];
        typename OV::Raw ov[KV];
    };
    auto geometry = [&](Tile &T, int blk) {
        T.g = block_group(sch, blk);
        T.lgL = pick(sch.log2_lanes, T.g);
        T.L = 1 << T.lgL;
        T.lb = pick(bins.log2b, T.g);
        T.nblk = int(pick(bins.nblk, T.g));
        const int64_t rows = pick(bins.rows, T.g);
        const int64_t first_row = pick(bins.first_row, T.g);
        T.vec_path = pick(sch.vec, T.g) == VEC;
        T.whole = T.nblk % VEC == 0 && pick(bins.first_elem, T.g) % VEC == 0;
        const int64_t tile = int64_t(blk - block_begin_of(sch, T.g)) * kSpmvWaves + wave;
        const int64_t row = (tile << (6 - T.lgL)) + (lane >> T.lgL);
        T.row_ok = row < rows;
        const int64_t row_c = T.row_ok ? row : rows - 1;
        T.sub = lane & (T.L - 1);
        T.j0 = row_c * T.nblk;                            // the row's first slot in its group
        T.e0 = pick(bins.first_elem, T.g) + T.j0;
        T.nvec = T.vec_path ? T.nblk / VEC : T.nblk;
        T.go = group_offsets(offs, bins, T.g);
        T.dest = perm[first_row + row_c];
        T.vrow = reinterpret_cast<const typename WV::V *>(values + T.e0);
    };
    auto issue = [&](Tile &T) {
        if (T.vec_path) {
#pragma unroll
            for (int t = 0; t < KV; ++t) {
                if (t * T.L < T.nvec) {                  // wave-uniform
                    const int vi = T.sub + t * T.L;
                    const int vc = vi < T.nvec ? vi : T.nvec - 1;
                    T.wv[t] = __builtin_nontemporal_load(T.vrow + vc);
                    T.ov[t] = OV::load(T.go, T.j0 + int64_t(vc) * VEC);
                }
            }
        }
        // INT8: the row's scale, loaded once its index has arrived (the vector loads
        // are already on their way)
        T.scale = kScaled<Tw> ? scales[T.dest] : 1.0f;
    };
    auto xat = [&](int c) -> float {
        // offsets from the encode always give c < N; the global path clamps anyway
        // so a malformed offset cannot read outside x
        if constexpr (LDS) return xs[c];
        else return to_f32<Tx>(x[c < N ? c : N - 1]);
    };
    auto finish = [&](Tile &T) {
        float acc = 0.0f;
        if (T.vec_path) {
            for (int base = 0;; base += T.L * KV) {
#pragma unroll
                for (int t = 0; t < KV; ++t) {
                    const int vi = base + T.sub + t * T.L;
                    if (vi < T.nvec) {
                        const typename OV::Bits ob = OV::bits(T.ov[t], T.go);
#pragma unroll
                        for (int q = 0; q < VEC; ++q) {
                            const int c = ((vi * VEC + q) << T.lb) + OV::field(ob, q, T.go);
                            acc = fmaf(WV::get(T.wv[t], q), xat(c), acc);
                        }
                    }
                }
                if (base + T.L * KV >= T.nvec) break;
#pragma unroll
                for (int t = 0; t < KV; ++t) {
                    if (base + T.L * KV + t * T.L < T.nvec) {   // wave-uniform
                        const int vi = base + T.L * KV + T.sub + t * T.L;
                        const int vc = vi < T.nvec ? vi : T.nvec - 1;
                        T.wv[t] = __builtin_nontemporal_load(T.vrow + vc);
                        T.ov[t] = OV::load(T.go, T.j0 + int64_t(vc) * VEC);
                    }
                }
            }
        } else if (T.whole) {
            // the vector path's order with element loads (a pointer not aligned for
            // vectors): lane sub takes vectors sub, sub + L, ..., each element in turn
            const Tw *vr = values + T.e0;
            for (int vi = T.sub; vi < T.nblk / VEC; vi += T.L) {
#pragma unroll
                for (int q = 0; q < VEC; ++q) {
                    const int k = vi * VEC + q;
                    const int o = OS::field(OS::bits(OS::load(T.go, T.j0 + k), T.go), 0, T.go);
                    acc = fmaf(to_f32<Tw>(vr[k]), xat((k << T.lb) + o), acc);
                }
            }
        } else {
            const Tw *vr = values + T.e0;
            for (int k = T.sub; k < T.nblk; k += T.L) {
                const int o = OS::field(OS::bits(OS::load(T.go, T.j0 + k), T.go), 0, T.go);
                acc = fmaf(to_f32<Tw>(vr[k]), xat((k << T.lb) + o), acc);
            }
        }
        acc = group_sum(acc, T.lgL);
        if (T.row_ok && T.sub == T.L - 1) y[T.dest] = kScaled<Tw> ? acc * T.scale : acc;
    };

    // The output row's index, then x's loads, then the first block's vectors: the
    // staging's memory latency overlaps the format's instead of queueing behind it.
    constexpr bool kDirect = SB == 0 && std::is_same<Tx, float>::value;  // fp32 x, 16 B aligned
    XStage<Tx, (SB > 0 ? SB : 1)> xst;
    Tile A;
    int blk = int(blockIdx.x);
    geometry(A, blk);
    if constexpr (LDS) {
        if constexpr (kDirect) stage_x_direct(xs, x, N);
        else xst.issue(x, N);
    }
    issue(A);
    if constexpr (LDS) {
        if constexpr (kDirect) {
            stage_x_tail(xs, x, N);
            __builtin_amdgcn_s_waitcnt(0);                 // the direct loads have landed
        } else {
            xst.commit(xs, x, N);
        }
        __syncthreads();
    }
    if constexpr (!LOOP) {
        finish(A);
    } else {
        // software pipelined over the workgroup's blocks: the next block's loads are
        // on their way while this one is summed
        Tile B;
        auto step = [&](Tile &cur, Tile &nxt) -> bool {
            const int nb = blk + int(gridDim.x);
            const bool more = nb < total_blocks;           // uniform
            if (more) {
                geometry(nxt, nb);
                issue(nxt);
            }
            finish(cur);
            blk = nb;
            return more;
        };
        for (;;) {
            if (!step(A, B)) break;
            if (!step(B, A)) break;
        }
    }
}

// ---------------------------------------------------------------------------------
// SpMV by row blocks: a block is four waves' tiles of rows of one group; workgroup
// (bx, g) takes blocks bx, bx + stride_g, ... of group g (blockIdx.y = g), so a
// wave's geometry needs no search.  Every input of the launch arrives with one round
// of scalar loads (the 64-byte header, the group's stride and its 32-byte record),
// issued by hand: a workgroup's first vector load waits on that round only.  Each
// wave loads its output row's index, then its share of x into LDS, then all its
// vectors; before the barrier it waits only until its share of x has landed (the
// vector loads return in order after it), so no wave waits for another wave's format
// data.  With one block per workgroup (LOOP false) the launch is one pass; with
// LOOP, workgroups stay resident, x is staged once, and each wave goes through its
// blocks load, wait, sum: the other waves of the CU hide its latency, and the next
// block's row index is loaded a block ahead so that the INT8 scale load never waits
// on a dependent round trip.
// ---------------------------------------------------------------------------------

struct SpmvRowsGroup {
    int32_t geo;          // nvec << 8 | lgL << 3 | lb: vectors per row, log2 lanes per row, log2 b
    int32_t rows;         // rows of the group
    int32_t first_row;    // storage index of the group's first row
    int32_t blocks;       // workgroups that hold rows (blockIdx.x < blocks)
    int64_t first_elem;   // slot of the group's first retained weight
    int64_t first_word;   // packed offsets: the group's first 32-bit word
};
struct SpmvRowsArgs {
    const void *values;
    const void *offs;     // byte offsets or packed words
    const void *x;
    float *y;
    const int32_t *perm;
    const float *scales;  // INT8 weights only
    int32_t N, pad[3];
    int32_t stride[kMaxBins];   // workgroups of group g: each takes blocks bx, bx + stride, ...
    SpmvRowsGroup g[kMaxBins];
};
static_assert(sizeof(SpmvRowsGroup) == 32, "group record is one 32-byte scalar load");
static_assert(offsetof(SpmvRowsArgs, stride) == 64, "header is one 64-byte scalar load");
static_assert(offsetof(SpmvRowsArgs, g) == 96, "group records follow the strides");


// s_waitcnt vmcnt(n): wait until at most n vector memory loads are outstanding
__device__ __forceinline__ void wait_vmcnt_le(int n) {
#define DARB_VMCNT(N)                                                                       \
    case N:                                                                                 \
        __builtin_amdgcn_s_waitcnt(0x0F70 | ((N) & 15) | ((((N) >> 4) & 3) << 14));         \
        break;
    switch (n) {
        DARB_VMCNT(0) DARB_VMCNT(1) DARB_VMCNT(2) DARB_VMCNT(3) DARB_VMCNT(4) DARB_VMCNT(5)
        DARB_VMCNT(6) DARB_VMCNT(7) DARB_VMCNT(8) DARB_VMCNT(9) DARB_VMCNT(10) DARB_VMCNT(11)
        DARB_VMCNT(12) DARB_VMCNT(13) DARB_VMCNT(14) DARB_VMCNT(15) DARB_VMCNT(16)
        DARB_VMCNT(17) DARB_VMCNT(18) DARB_VMCNT(19) DARB_VMCNT(20)
        default: __builtin_amdgcn_s_waitcnt(0x0F70); break;       // vmcnt(0)
    }
#undef DARB_VMCNT
}

template <typename Tw, typename Tx, int KV, bool PK, bool LOOP>
__global__ __launch_bounds__(kSpmvThreads, 4) void spmv_rows_kernel(SpmvRowsArgs args) {
    using WV = WVec<Tw>;
    constexpr int VEC = WV::VEC;
    using OV = Off<PK, VEC>;
    constexpr int XB = int(sizeof(Tx));                      // bytes per element of x
    constexpr int LGXB = XB == 4 ? 2 : 1;
    extern __shared__ float xs[];                             // x as stored (Tx), then a pad
    (void)args;   // read below through the kernel-argument segment

    typedef int i32x16 __attribute__((ext_vector_type(16)));
    typedef int i32x8 __attribute__((ext_vector_type(8)));
    i32x16 H;
    i32x8 Gr;
    int stride;
    {
        const auto kp = __builtin_amdgcn_kernarg_segment_ptr();
        const uint32_t goff = uint32_t(offsetof(SpmvRowsArgs, g)) +
                              uint32_t(sizeof(SpmvRowsGroup)) * blockIdx.y;
        const uint32_t soff = uint32_t(offsetof(SpmvRowsArgs, stride)) + 4u * blockIdx.y;
        asm volatile("s_load_dwordx16 %0, %3, 0x0\n\t"
                     "s_load_dwordx8 %1, %3, %4\n\t"
                     "s_load_dword %2, %3, %5\n\t"
                     "s_waitcnt lgkmcnt(0)"
                     : "=s"(H), "=s"(Gr), "=s"(stride) : "s"(kp), "s"(goff), "s"(soff) : "memory");
    }
    // the pointers are global memory: built as global pointers so that every access
    // through them is a global (not flat) instruction
    typedef __attribute__((address_space(1))) char gchar;
    auto ptr = [&](int i) -> void * {
        return (void *)(gchar *)(uintptr_t((uint64_t(uint32_t(H[2 * i + 1])) << 32) |
                                           uint32_t(H[2 * i])));
    };
    const Tw *values = static_cast<const Tw *>(ptr(0));
    const void *offs = ptr(1);
    const char *x = static_cast<const char *>(ptr(2));
    float *y = static_cast<float *>(ptr(3));
    const int32_t *perm = static_cast<const int32_t *>(ptr(4));
    const float *scales = static_cast<const float *>(ptr(5));
    const int N = H[12];
    const int geo = Gr[0], rows = Gr[1], first_row = Gr[2], blocks = Gr[3];
    const int64_t first_elem = int64_t((uint64_t(uint32_t(Gr[5])) << 32) | uint32_t(Gr[4]));
    const int64_t first_word = int64_t((uint64_t(uint32_t(Gr[7])) << 32) | uint32_t(Gr[6]));
    // uniform: a group with fewer blocks, or fewer resident workgroups, than the grid row
    if (int(blockIdx.x) >= blocks || int(blockIdx.x) >= stride) return;

    const int wave = wave_uniform(int(threadIdx.x) / kWave);
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int lb = geo & 7, lgL = (geo >> 3) & 7, nvec = geo >> 8;
    const int L = 1 << lgL;
    const int sub = lane & (L - 1);
    const int n = (nvec + L - 1) >> lgL;                     // vectors per lane (uniform)
    // the lane's row in block blk (clamped into the group) and whether it exists
    auto row_of = [&](int blk, bool &ok) {
        const int row = ((blk * kSpmvWaves + wave) << (6 - lgL)) + (lane >> lgL);
        ok = row < rows;
        return ok ? row : rows - 1;
    };
    int blk = int(blockIdx.x);
    bool row_ok;
    int row_c = row_of(blk, row_ok);
    int32_t dest = perm[first_row + row_c];

    // x into LDS as stored, by DMA in 1 KiB chunks (x is 16-byte aligned and a whole
    // number of 16-byte vectors); the last chunk's lanes past x's end repeat x's last
    // vector into the pad.  No LDS store follows, so nothing waits for all of it.
    {
        typedef __attribute__((address_space(1))) const char *gptr;
        typedef __attribute__((address_space(3))) void *lptr;
        const int nv16 = (N * XB) >> 4;
        const int chunks = (nv16 + kWave - 1) / kWave;
        for (int j = wave; j < chunks; j += kSpmvWaves) {
            const int v = j * kWave + lane;
            __builtin_amdgcn_global_load_lds((gptr)(x + (v < nv16 ? v : nv16 - 1) * 16),
                                             (lptr)(reinterpret_cast<char *>(xs) + j * kWave * 16),
                                             16, 0, 0);
        }
    }

    GroupOffsets go;
    go.u8 = static_cast<const uint8_t *>(offs) + first_elem;
    go.pk = packed_group(static_cast<const uint32_t *>(offs), first_word, lb);
    // vectors a lane loads: its n, or all KV when KV is small (a fixed count keeps the
    // compiler from copying vectors between branches, which would wait on the loads)
    constexpr bool kAll = KV <= 4;
    const int nl = kAll ? KV : n;
    typename WV::V wv[KV];
    typename OV::Raw ov[KV];
    auto load_block = [&](int rc) {
        const int64_t j0 = int64_t(rc) * (int64_t(nvec) * VEC);   // the row's first slot in its group
        const typename WV::V *vrow =
            reinterpret_cast<const typename WV::V *>(values + first_elem + j0);
#pragma unroll
        for (int k = 0; k < KV; ++k) {
            if (kAll || k < n) {                             // uniform
                // keeps the loads inside the branch: issued unconditionally they would
                // cost load slots for nothing
                if constexpr (!kAll) asm volatile("" ::: "memory");
                int vi = sub + k * L;
                vi = vi < nvec ? vi : nvec - 1;
                wv[k] = __builtin_nontemporal_load(vrow + vi);
                ov[k] = OV::load(go, j0 + int64_t(vi) * VEC);
            }
        }
    };
    // the sums of one block: block size b = 2^LB fixed at compile time, so each
    // gather's in-block position is an immediate of its LDS load and an offset costs one
    // extract and one add
    auto sum_block = [&](float scale, bool ok, int32_t d, auto lbc) {
        constexpr int LB = decltype(lbc)::value;
        constexpr uint32_t sh = uint32_t(LB + LGXB);
        const uint32_t base = uint32_t(sub * VEC) << sh;     // byte address of the lane's first block
        const uint32_t stepk = uint32_t(L * VEC) << sh;
        const uint32_t lastb = uint32_t((nvec - 1) * VEC) << sh;
        float acc = 0.0f;
#pragma unroll
        for (int k = 0; k < KV; ++k) {
            if (k < n) {
                uint32_t bk = base + uint32_t(k) * stepk;
                bk = bk < lastb ? bk : lastb;
                const typename OV::Bits ob = OV::bits(ov[k], go);
                float xv[VEC];
#pragma unroll
                for (int q = 0; q < VEC; ++q) {
                    const uint32_t ad = bk + (uint32_t(OV::template field_c<LB>(ob, q)) << LGXB);
                    xv[q] = to_f32<Tx>(*reinterpret_cast<const Tx *>(
                        reinterpret_cast<const char *>(xs) + ad + (uint32_t(q) << sh)));
                }
                if (sub + k * L < nvec) {
#pragma unroll
                    for (int q = 0; q < VEC; ++q) acc = fmaf(WV::get(wv[k], q), xv[q], acc);
                }
            }
        }
        acc = group_sum(acc, lgL);
        if (ok && sub == L - 1) y[d] = kScaled<Tw> ? acc * scale : acc;
    };

    load_block(row_c);
    // INT8: the row's scale, once its index has arrived (the loads above are on their way)
    float scale = 1.0f;
    asm volatile("" ::: "memory");
    if constexpr (kScaled<Tw>) scale = scales[dest];
    // loads return in order: at most (vector loads + scale load) outstanding means this
    // wave's x chunks have landed; every vector issues at least two loads
    wait_vmcnt_le(2 * nl + (kScaled<Tw> ? 1 : 0));
    asm volatile("s_barrier" ::: "memory");
    auto sum_any = [&](float sc, bool ok, int32_t d) {
        switch (lb) {                                        // uniform
            case 0: sum_block(sc, ok, d, std::integral_constant<int, 0>{}); break;
            case 1: sum_block(sc, ok, d, std::integral_constant<int, 1>{}); break;
            case 2: sum_block(sc, ok, d, std::integral_constant<int, 2>{}); break;
            case 3: sum_block(sc, ok, d, std::integral_constant<int, 3>{}); break;
            case 4: sum_block(sc, ok, d, std::integral_constant<int, 4>{}); break;
            case 5: sum_block(sc, ok, d, std::integral_constant<int, 5>{}); break;
            case 6: sum_block(sc, ok, d, std::integral_constant<int, 6>{}); break;
            default: sum_block(sc, ok, d, std::integral_constant<int, 7>{}); break;
        }
    };
    if constexpr (!LOOP) {
        sum_any(scale, row_ok, dest);
    } else {
        for (;;) {
            const int nxt = blk + stride;
            const bool more = nxt < blocks;                  // uniform
            bool nok = false;
            int nrc = 0;
            int32_t ndest = 0;
            if (more) {
                nrc = row_of(nxt, nok);
                ndest = perm[first_row + nrc];               // one block ahead
            }
            sum_any(scale, row_ok, dest);
            if (!more) break;
            blk = nxt;
            row_ok = nok;
            dest = ndest;
            load_block(nrc);
            if constexpr (kScaled<Tw>) scale = scales[dest];
        }
    }
}

// ---------------------------------------------------------------------------------
// SpMM
// ---------------------------------------------------------------------------------

constexpr int kSpmmThreads = 512;
constexpr int kSpmmWaves = kSpmmThreads / kWave;
constexpr int kSpmmBatch = 8;         // X rows in flight per lane (more waves beat deeper batches)
constexpr int kRowLanes = 16;         // lanes per row that narrow columns aim at

// CPL consecutive batch columns of one X row, loaded at once (16 bytes when CPL > 1).
template <typename Tx, int CPL> struct XLoad;
template <typename Tx> struct XLoad<Tx, 1> {
    using V = Tx;
    __device__ static V load(const Tx *p) { return *p; }
    __device__ static float get(const V &v, int) { return to_f32<Tx>(v); }
};
template <> struct XLoad<float, 4> {
    using V = f32x4;
    __device__ static V load(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }
    __device__ static float get(const V &v, int i) { return v[i]; }
};
template <> struct XLoad<float, 2> {
    using V = f32x2;
    __device__ static V load(const float *p) { return *reinterpret_cast<const f32x2 *>(p); }
    __device__ static float get(const V &v, int i) { return v[i]; }
};
template <> struct XLoad<__half, 2> {
    using V = uint32_t;
    __device__ static V load(const __half *p) { return *reinterpret_cast<const uint32_t *>(p); }
    __device__ static float get(const V &v, int i) { return half_bits_to_f32(i ? v >> 16 : v); }
};
template <> struct XLoad<__half, 4> {
    using V = u32x2;
    __device__ static V load(const __half *p) { return *reinterpret_cast<const u32x2 *>(p); }
    __device__ static float get(const V &v, int i) {
        const uint32_t w = v[i >> 1];
        return half_bits_to_f32((i & 1) ? (w >> 16) : w);
    }
};
template <> struct XLoad<__half, 8> {
    using V = u32x4;
    __device__ static V load(const __half *p) { return *reinterpret_cast<const u32x4 *>(p); }
    __device__ static float get(const V &v, int i) {
        const uint32_t w = v[i >> 1];
        return half_bits_to_f32((i & 1) ? (w >> 16) : w);
    }
};

template <int Base, typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, Is...>) {
    (f(std::integral_constant<int, Base + Is>{}), ...);
}
// f(integral_constant<int, i>) for i = Base .. Base + Count - 1, unrolled at compile time
template <int Base, int Count, typename F> __device__ __forceinline__ void static_for(F &&f) {
    static_for_impl<Base>(f, std::make_integer_sequence<int, Count>{});
}

// Value of lane T of the caller's group of 2^LGL consecutive lanes, for every lane
// of the group (T is a compile-time lane index inside the group).
template <int LGL, int T> __device__ __forceinline__ int group_bcast(int v) {
    if constexpr (LGL == 0) {
        return v;
    } else if constexpr (LGL == 1) {                      // DPP quad_perm [T, T, 2+T, 2+T]
        return __builtin_amdgcn_update_dpp(0, v, T | (T << 2) | ((2 + T) << 4) | ((2 + T) << 6),
                                           0xF, 0xF, false);
    } else if constexpr (LGL == 2) {                      // DPP quad_perm [T, T, T, T]
        return __builtin_amdgcn_update_dpp(0, v, T * 0x55, 0xF, 0xF, false);
    } else if constexpr (LGL == 4) {                      // DPP row_newbcast:T (16-lane rows)
        return __builtin_amdgcn_update_dpp(0, v, 0x150 + T, 0xF, 0xF, false);
    } else if constexpr (LGL == 6) {                      // whole wave: through a scalar register
        return __builtin_amdgcn_readlane(v, T);
    } else {                                              // 8 or 32 lanes: ds_swizzle bitmask mode
        constexpr int and_mask = 0x1F & ~((1 << LGL) - 1);
        return __builtin_amdgcn_ds_swizzle(v, (T << 5) | and_mask);
    }
}

// GM consecutive retained weights of a row (values and offsets) for one lane: one
// vector load each when the bin is aligned for it, element loads otherwise.
template <typename Tw, int GM, bool PK> struct PairLoad {
    struct alignas(GM * sizeof(Tw)) VV { Tw e[GM]; };
    using OV = Off<PK, GM>;
    // the vector form as loaded, kept in registers while other loads are in flight
    struct Raw { VV a; typename OV::Raw ob; };
    // vec: the caller guarantees k % GM == 0, k + GM <= nblk and nblk % GM == 0 (so
    // the group slot j0 + k is a multiple of GM); otherwise every element index is
    // clamped into the row [0, nblk).  j0 is the row's first slot in its group.
    __device__ static Raw issue(const Tw *vr, const GroupOffsets &go, int64_t j0, int k) {
        return Raw{*reinterpret_cast<const VV *>(vr + k), OV::load(go, j0 + k)};
    }
    __device__ static void decode(const Raw &r, const GroupOffsets &go, float (&v)[GM],
                                  int (&o)[GM]) {
        const typename OV::Bits b = OV::bits(r.ob, go);
#pragma unroll
        for (int i = 0; i < GM; ++i) {
            v[i] = to_f32<Tw>(r.a.e[i]);
            o[i] = OV::field(b, i, go);
        }
    }
    __device__ static void load(const Tw *vr, const GroupOffsets &go, int64_t j0, int k,
                                int nblk, bool vec, float (&v)[GM], int (&o)[GM]) {
        if (vec) {
            decode(issue(vr, go, j0, k), go, v, o);
        } else {
            using OS = Off<PK, 1>;
#pragma unroll
            for (int i = 0; i < GM; ++i) {
                const int kk = k + i < nblk ? k + i : nblk - 1;
                v[i] = to_f32<Tw>(vr[kk]);
                o[i] = OS::field(OS::bits(OS::load(go, j0 + kk), go), 0, go);
            }
        }
    }
};

// One workgroup-sized tile of the SpMM: lanes map to batch columns (CPL per lane,
// 2^LGL lanes per matrix row, 64 >> LGL rows per wave).  A wave owns a contiguous
// share [kbeg, kend) of its rows' weights (KS waves split a row group).  The lanes
// of a row load S = max(2^LGL, 16) of the row's (value, column) pairs per step, one
// pair per lane and group, straight from HBM with coalesced loads, then broadcast
// each pair to the row's lanes with a register-to-register exchange and gather its
// X row; kSpmmBatch gathers are in flight per lane.  With aligned pairs the loads
// are software pipelined: a round's pairs are issued right after the previous
// round's last gathers, so their HBM latency overlaps those gathers.  Partial sums
// of the KS waves meet in LDS (`part`, kSpmmThreads * CPL floats) in a fixed order.
// The finished rows go to
//     epi(row_ok, col_ok, original row, first column, acc[CPL], lane in row),
// called by every lane of the waves that hold finished rows (wave-uniform), so an
// epilogue may exchange values between the lanes of a row.
template <typename Tw, typename Tx, int CPL, int LGL, bool PK, typename Epi>
__device__ __forceinline__ void spmm_tile(
    int tile, const Tw *__restrict__ values, const void *__restrict__ offs,
    const Tx *__restrict__ X, int64_t ldx, int64_t B, const int32_t *__restrict__ perm, int N,
    const BinTable &bins, const ProductSchedule &sch, float *part, Epi &&epi) {
    using XL = XLoad<Tx, CPL>;
    constexpr int L = 1 << LGL;
    constexpr int R = kWave >> LGL;                       // rows per wave
    constexpr int GM = L >= 16 ? 1 : 16 / L;              // pair groups per lane per step
    constexpr int S = L * GM;                             // weights per row per step
    // steps whose pairs load together: four for rows of 16 or fewer lanes (measured
    // 11 % faster at 16 lanes, batch 64), two when the offsets are packed (their word
    // windows take more registers); a 64-lane row's step already spans 64 weights
    constexpr int DEPTH = (L >= kWave || GM >= 4) ? 1 : (PK ? 2 : 4) / GM;
    constexpr int T = DEPTH * S;                          // weights per row per round
    constexpr int NB = kSpmmBatch;                        // X-row gathers in flight per lane
    static_assert(S % NB == 0, "a gather batch lies inside one step");

    const int g = block_group(sch, tile);
    const int wave = wave_uniform(int(threadIdx.x) / kWave);
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int KS = pick(sch.ksplit, g);
    const int rows_pb = R * (kSpmmWaves / KS);
    const int lb = pick(bins.log2b, g);
    const int nblk = int(pick(bins.nblk, g));
    const int64_t rows = pick(bins.rows, g);
    const int64_t first_row = pick(bins.first_row, g);
    const int64_t first_elem = pick(bins.first_elem, g);

    // column slab outermost: the workgroups in flight together share one slab of X,
    // which stays in L2 even when all of X does not
    const int local = tile - block_begin_of(sch, g);
    const int row_blks = int((rows + rows_pb - 1) / rows_pb);
    const int slab = local / row_blks;
    const int row_blk = local - slab * row_blks;
    const int64_t row0 = int64_t(row_blk) * rows_pb;
    const int rows_here = int(rows - row0 < rows_pb ? rows - row0 : rows_pb);

    const int rg = wave / KS, ks = wave - (wave / KS) * KS;
    const int rl = rg * R + (lane >> LGL);                // row of this lane in the block
    const bool row_ok = rl < rows_here;
    const int sub = lane & (L - 1);
    const int64_t col0 = (int64_t(slab) * L + sub) * CPL;
    const bool col_ok = col0 < B;                         // CPL > 1 only when CPL divides B
    const int64_t col_c = col_ok ? col0 : 0;
    // each wave's share is a multiple of 16 weights (of GM, so a lane's GM-vector of
    // weights is either entirely inside [kbeg, kend) or entirely outside); the split
    // points do not depend on the lanes per row, so neither do the sums
    const int share = (((nblk + KS - 1) / KS) + 15) / 16 * 16;
    const int kbeg = ks * share;
    const int kend = kbeg + share < nblk ? kbeg + share : nblk;
    const int64_t j0 = (row0 + (row_ok ? rl : 0)) * nblk;   // the row's first slot in its group
    const Tw *vr = values + first_elem + j0;
    const GroupOffsets go = group_offsets(offs, bins, g);

    float acc[CPL];
#pragma unroll
    for (int q = 0; q < CPL; ++q) acc[q] = 0.0f;

    const bool vec_pairs = pick(sch.vec, g) != 0;
    using PL = PairLoad<Tw, GM, PK>;
    // a round's pairs (DEPTH steps) as values and clamped columns; -1 marks no weight
    auto settle = [&](int k0, int st, const float (&v)[GM], const int (&o)[GM],
                      float (&vl)[DEPTH][GM], int (&cl)[DEPTH][GM]) {
        const int k = k0 + st * S + sub * GM;
        const bool ok = row_ok && k < kend;
#pragma unroll
        for (int gi = 0; gi < GM; ++gi) {
            const bool okg = ok && k + gi < kend;         // element test for the scalar path
            vl[st][gi] = okg ? v[gi] : 0.0f;
            const int c = ((k + gi) << lb) + o[gi];
            cl[st][gi] = okg ? (c < N ? c : N - 1) : -1;   // the encode gives c < N
        }
    };
    // vector pair loads of the round at k0 (lanes past the share or the rows load a
    // valid slot of their row block and are masked when settled)
    auto issue_round = [&](int k0, typename PL::Raw (&raw)[DEPTH]) {
#pragma unroll
        for (int st = 0; st < DEPTH; ++st) {
            const int k = k0 + st * S + sub * GM;
            raw[st] = PL::issue(vr, go, j0, row_ok && k < kend ? k : kbeg);
        }
    };
    // gathers of one round (DEPTH steps of S weights), NB X rows in flight per lane;
    // `after` runs right after the round's last gathers are issued (the next round's
    // pair loads go there, so they overlap these gathers without delaying their use)
    auto gather_round = [&](int k0, const float (&vl)[DEPTH][GM], const int (&cl)[DEPTH][GM],
                            auto &&after) {
        static_for<0, T / NB>([&](auto bc) {
            constexpr int b0 = decltype(bc)::value * NB;
            if (k0 + (b0 / S) * S >= kend) return;         // wave-uniform: past the share
            float vv[NB];
            int cc[NB];
            typename XL::V xv[NB];
            static_for<0, NB>([&](auto uc) {
                constexpr int f = b0 + decltype(uc)::value;   // weight k0 + f of the round
                constexpr int st = f / S, fs = f % S;
                vv[f - b0] = __builtin_bit_cast(
                    float, group_bcast<LGL, fs / GM>(__builtin_bit_cast(int, vl[st][fs % GM])));
                cc[f - b0] = group_bcast<LGL, fs / GM>(cl[st][fs % GM]);
                const int64_t c = cc[f - b0] >= 0 ? cc[f - b0] : 0;
                xv[f - b0] = XL::load(X + c * ldx + col_c);
            });
            if constexpr (b0 + NB == T) after();
#pragma unroll
            for (int u = 0; u < NB; ++u) {
                if (cc[u] >= 0 && col_ok) {
#pragma unroll
                    for (int q = 0; q < CPL; ++q)
                        acc[q] = fmaf(vv[u], XL::get(xv[u], q), acc[q]);
                }
            }
        });
    };

    if (vec_pairs) {
        // software pipelined: the pairs of round i + 1 load while round i gathers
        typename PL::Raw raw[DEPTH];
        if (kbeg < kend) issue_round(kbeg, raw);          // wave-uniform
        for (int k0 = kbeg; k0 < kend; k0 += DEPTH * S) {
            float vl[DEPTH][GM];
            int cl[DEPTH][GM];
#pragma unroll
            for (int st = 0; st < DEPTH; ++st) {
                float v[GM];
                int o[GM];
                PL::decode(raw[st], go, v, o);
                settle(k0, st, v, o, vl, cl);
            }
            const int k1 = k0 + DEPTH * S;
            gather_round(k0, vl, cl, [&] {
                if (k1 < kend) issue_round(k1, raw);      // wave-uniform
            });
        }
    } else {
        for (int k0 = kbeg; k0 < kend; k0 += DEPTH * S) {
            float vl[DEPTH][GM];
            int cl[DEPTH][GM];
#pragma unroll
            for (int st = 0; st < DEPTH; ++st) {
                const int k = k0 + st * S + sub * GM;
                float v[GM];
                int o[GM];
                PL::load(vr, go, j0, row_ok && k < kend ? k : kbeg, nblk, false, v, o);
                settle(k0, st, v, o, vl, cl);
            }
            gather_round(k0, vl, cl, [] {});
        }
    }

    // combine the KS partial sums of each row group in a fixed order
    if (KS > 1) {
#pragma unroll
        for (int q = 0; q < CPL; ++q) part[(wave * kWave + lane) * CPL + q] = acc[q];
        __syncthreads();
        if (ks == 0) {
            for (int s2 = 1; s2 < KS; ++s2) {
#pragma unroll
                for (int q = 0; q < CPL; ++q)
                    acc[q] += part[((wave + s2) * kWave + lane) * CPL + q];
            }
        }
    }
    if (ks == 0) epi(row_ok, col_ok, row_ok ? perm[first_row + row0 + rl] : 0, col0, acc, sub);
}

template <typename Tw, typename Tx, int CPL, int LGL, bool PK>
__global__ __launch_bounds__(kSpmmThreads) void spmm_kernel(
    const Tw *__restrict__ values, const void *__restrict__ offs,
    const Tx *__restrict__ X, int64_t ldx, int64_t B, float *__restrict__ Y, int64_t ldy,
    const int32_t *__restrict__ perm, int N, BinTable bins, ProductSchedule sch,
    const float *__restrict__ scales) {
    __shared__ float part[kSpmmThreads * CPL];
    spmm_tile<Tw, Tx, CPL, LGL, PK>(
        int(blockIdx.x), values, offs, X, ldx, B, perm, N, bins, sch, part,
        [&](bool row_ok, bool col_ok, int32_t orig, int64_t col0, const float (&acc)[CPL], int) {
            if (row_ok && col_ok) {
                const float sc = kScaled<Tw> ? scales[orig] : 1.0f;
                float *yrow = Y + int64_t(orig) * ldy + col0;
#pragma unroll
                for (int q = 0; q < CPL; ++q) yrow[q] = kScaled<Tw> ? acc[q] * sc : acc[q];
            }
        });
}

// ---------------------------------------------------------------------------------
// SpMM for short rows of X and many batch columns (the recurrent workload's input
// products: N = 1024, B = 6400).  A workgroup takes one slab of SC = 4L batch
// columns, copies X[:, slab] (N x SC fp32, <= 128 KiB) into LDS once, then runs
// every row of every group against it -- the X-row gathers hit LDS instead of L2.
// The format is read by every workgroup, from L2.  One lane group of L lanes per
// row; each lane loads a step's 16 (value, offset) pairs itself (offsets as bytes
// or as packed words: the same sums either way), the next step's while this one
// gathers.
// ---------------------------------------------------------------------------------

constexpr int kXldsThreads = 1024;
constexpr int kXldsWaves = kXldsThreads / kWave;
constexpr int kXldsFloats = 32768;                  // 128 KiB of LDS
constexpr int kXldsStep = 16;                       // weights per row per step
constexpr int kXldsBatch = 16;                      // LDS gathers in flight per lane

// 16 consecutive retained values of one row, loaded as 16-byte vectors (load) or
// element by element from any alignment (load_elem), to the same registers.
template <typename Tw> struct Step16;
template <> struct Step16<float> {
    f32x4 v[4];
    __device__ static Step16 load(const float *p) {
        Step16 s;
#pragma unroll
        for (int i = 0; i < 4; ++i) s.v[i] = reinterpret_cast<const f32x4 *>(p)[i];
        return s;
    }
    __device__ static Step16 load_elem(const float *p) {
        Step16 s;
#pragma unroll
        for (int i = 0; i < 16; ++i) s.v[i >> 2][i & 3] = p[i];
        return s;
    }
    __device__ float get(int i) const { return v[i >> 2][i & 3]; }
};
template <> struct Step16<__half> {
    u32x4 v[2];
    __device__ static Step16 load(const __half *p) {
        Step16 s;
#pragma unroll
        for (int i = 0; i < 2; ++i) s.v[i] = reinterpret_cast<const u32x4 *>(p)[i];
        return s;
    }
    __device__ static Step16 load_elem(const __half *p) {
        const uint16_t *h = reinterpret_cast<const uint16_t *>(p);
        Step16 s;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            s.v[i >> 2][i & 3] = uint32_t(h[2 * i]) | (uint32_t(h[2 * i + 1]) << 16);
        return s;
    }
    __device__ float get(int i) const {
        const uint32_t w = v[i >> 3][(i >> 1) & 3];
        return half_bits_to_f32((i & 1) ? (w >> 16) : w);
    }
};

// ELEM: values or byte offsets not 16-byte aligned, loaded element by element (the
// same registers, so the same sums); xvec: X's rows 16-byte aligned and B a multiple
// of 4 (staged as 16-byte vectors, otherwise element by element).
template <typename Tw, int LGL, bool PK, bool ELEM>
__global__ __launch_bounds__(kXldsThreads) void spmm_xlds_kernel(
    const Tw *__restrict__ values, const void *__restrict__ offs,
    const float *__restrict__ X, int64_t ldx, int64_t B, float *__restrict__ Y, int64_t ldy,
    const int32_t *__restrict__ perm, int N, BinTable bins, ProductSchedule sch, bool xvec) {
    constexpr int L = 1 << LGL;
    constexpr int R = kWave >> LGL;
    constexpr int SC = 4 * L;                           // slab columns
    constexpr int kStage = 8;                           // 16-byte staging loads in flight
    __shared__ float xs[kXldsFloats];
    using XL = XLoad<float, 4>;
    using OV = Off<PK, kXldsStep>;                      // a step's 16 offsets

    const int64_t colbase = int64_t(blockIdx.x) * SC;
    // X[:, slab] -> xs[c * SC + j]; columns past B read as zero
    if (xvec) {                                         // uniform: 4 divides B
        constexpr int per_row = SC / 4;
        const int items = N * per_row;
        for (int base = 0; base < items; base += kStage * kXldsThreads) {
            f32x4 v[kStage];
            bool in[kStage];
#pragma unroll
            for (int u = 0; u < kStage; ++u) {
                const int i = base + u * kXldsThreads + int(threadIdx.x);
                const int ic = i < items ? i : items - 1;
                const int c = ic / per_row, q = ic - c * per_row;
                const int64_t col = colbase + int64_t(q) * 4;
                in[u] = i < items && col < B;
                v[u] = XL::load(X + int64_t(c) * ldx + (col < B ? col : 0));
            }
#pragma unroll
            for (int u = 0; u < kStage; ++u) {
                const int i = base + u * kXldsThreads + int(threadIdx.x);
                if (i < items) {
                    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
                    *reinterpret_cast<f32x4 *>(xs + i * 4) = in[u] ? v[u] : z;
                }
            }
        }
    } else {
        for (int i = int(threadIdx.x); i < N * SC; i += kXldsThreads) {
            const int c = i / SC, j = i - c * SC;
            const int64_t col = colbase + j;
            xs[i] = col < B ? X[int64_t(c) * ldx + col] : 0.0f;
        }
    }
    __syncthreads();
    // a step's 16 values and 16 offsets, as vectors or element by element
    auto load_w = [&](int64_t e) {
        if constexpr (ELEM) return Step16<Tw>::load_elem(values + e);
        else return Step16<Tw>::load(values + e);
    };
    auto load_o = [&](const GroupOffsets &go, int64_t j) {
        if constexpr (ELEM && !PK) {                    // 16 offset bytes, one at a time
            typename OV::Raw r;
#pragma unroll
            for (int wd = 0; wd < 4; ++wd) {
                uint32_t v = 0;
#pragma unroll
                for (int b = 0; b < 4; ++b) v |= uint32_t(go.u8[j + 4 * wd + b]) << (8 * b);
                r[wd] = v;
            }
            return r;
        } else {
            return OV::load(go, j);                     // packed words need no alignment
        }
    };

    const int wave = wave_uniform(int(threadIdx.x) / kWave);
    const int lane = int(threadIdx.x) & (kWave - 1);
    const int sub = lane & (L - 1);
    const int64_t col0 = colbase + int64_t(sub) * 4;
    const bool col_ok = col0 < B;
    const int xoff = sub * 4;
    for (int g = 0; g < sch.nbins; ++g) {                // uniform
        const int lb = pick(bins.log2b, g);
        const int nblk = int(pick(bins.nblk, g));        // a multiple of kXldsStep
        const int64_t rows = pick(bins.rows, g);
        const int64_t first_row = pick(bins.first_row, g);
        const int64_t first_elem = pick(bins.first_elem, g);
        const GroupOffsets go = group_offsets(offs, bins, g);
        for (int64_t p0 = 0; p0 < rows; p0 += int64_t(kXldsWaves) * R) {
            const int64_t rl = p0 + wave * R + (lane >> LGL);
            const bool row_ok = rl < rows;
            const int64_t j0 = (row_ok ? rl : 0) * nblk;   // the row's first slot, 16-aligned
            const int64_t e0 = first_elem + j0;
            float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            // every lane of the row loads the step's 16 (value, offset) pairs itself
            // (equal addresses within one load merge), so no lane exchange is needed;
            // the next step's pairs load while this step gathers
            Step16<Tw> w = load_w(e0);
            typename OV::Raw ob = load_o(go, j0);
            for (int k0 = 0; k0 < nblk; k0 += kXldsStep) {
                const int kn = k0 + kXldsStep < nblk ? k0 + kXldsStep : k0;
                const Step16<Tw> w_next = load_w(e0 + kn);
                const typename OV::Raw ob_next = load_o(go, j0 + kn);
                const typename OV::Bits obits = OV::bits(ob, go);
                static_for<0, kXldsStep / kXldsBatch>([&](auto bc) {
                    constexpr int b0 = decltype(bc)::value * kXldsBatch;
                    f32x4 xv[kXldsBatch];
                    static_for<0, kXldsBatch>([&](auto uc) {
                        constexpr int f = b0 + decltype(uc)::value;
                        const int o = OV::field(obits, f, go);
                        int c = ((k0 + f) << lb) + o;
                        c = c < N ? c : N - 1;                // the encode gives c < N
                        xv[f - b0] = *reinterpret_cast<const f32x4 *>(xs + c * SC + xoff);
                    });
#pragma unroll
                    for (int u = 0; u < kXldsBatch; ++u) {
                        const float vw = w.get(b0 + u);
#pragma unroll
                        for (int q = 0; q < 4; ++q) acc[q] = fmaf(vw, xv[u][q], acc[q]);
                    }
                });
                w = w_next;
                ob = ob_next;
            }
            if (row_ok && col_ok) {
                float *yrow = Y + int64_t(perm[first_row + rl]) * ldy + col0;
                if (col0 + 3 < B) {                      // a whole quad: one 16-byte store
                    typedef float f32x4_u __attribute__((ext_vector_type(4), aligned(4)));
                    *reinterpret_cast<f32x4_u *>(yrow) = f32x4_u{acc[0], acc[1], acc[2], acc[3]};
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (col0 + q < B) yrow[q] = acc[q];
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------------
// host-side schedules and launches
// ---------------------------------------------------------------------------------

inline int ilog2_ceil(int64_t v) {
    int l = 0;
    while ((int64_t(1) << l) < v) ++l;
    return l;
}

// The offsets argument of the kernels: the byte form, or the packed words.  A plan
// without packed words has b = 1 everywhere; the kernels then still load one word
// (and mask it to nothing), so they get the plan's row order, >= 4 readable bytes.
inline const void *offset_source(const darb_plan &p, const uint8_t *offsets,
                                 const uint32_t *packed) {
    if (offsets) return offsets;
    return p.packed_words > 0 ? static_cast<const void *>(packed)
                              : static_cast<const void *>(p.d_perm);
}

// Byte offsets are loaded VEC at a time, so their address must be aligned for it;
// packed offsets are loaded as whole words at any weight index.
inline bool offsets_aligned(const uint8_t *offsets, int vec) {
    return !offsets || reinterpret_cast<uintptr_t>(offsets) % vec == 0;
}

// vmax: vectors per lane the lanes-per-row choice aims at (<= kVmax)
template <typename Tw>
bool spmv_schedule(const darb_plan &p, const void *values, const uint8_t *offsets,
                   ProductSchedule &s, int vmax = kVmax) {
    constexpr int VEC = WVec<Tw>::VEC;
    s = ProductSchedule{};
    s.nbins = p.bins.nbins;
    s.col_slabs = 1;
    const bool ptr_ok =
        (reinterpret_cast<uintptr_t>(values) % sizeof(typename WVec<Tw>::V) == 0) &&
        offsets_aligned(offsets, VEC);
    int64_t blocks = 0;
    for (int g = 0; g < s.nbins; ++g) {
        const int64_t nblk = p.bins.nblk[g];
        // rows of whole vectors split into vectors whatever the pointers' alignment
        // (which only chooses vector or element loads), so every path sums a row in
        // the same order and gives the same bits
        const bool whole = nblk % VEC == 0 && p.bins.first_elem[g] % VEC == 0;
        s.vec[g] = ptr_ok && whole ? VEC : 1;
        const int64_t nvec = whole ? nblk / VEC : nblk;
        int lgL = 0;     // fewest lanes per row that keep each lane within vmax vectors
        while (lgL < 6 && ((nvec + (int64_t(1) << lgL) - 1) >> lgL) > vmax) ++lgL;
        s.log2_lanes[g] = lgL;
        s.block_begin[g] = int32_t(blocks);
        const int64_t rows_per_wave = int64_t(kWave) >> lgL;
        const int64_t tiles = (p.bins.rows[g] + rows_per_wave - 1) / rows_per_wave;
        blocks += (tiles + kSpmvWaves - 1) / kSpmvWaves;
        if (blocks > 0x7FFFFFFF) return false;
    }
    s.block_begin[s.nbins] = int32_t(blocks);
    return true;
}

// The row-block kernel when it applies: x is 16-byte aligned, a whole number of
// 16-byte vectors and fits in 64 KiB of LDS with its pad, and every group takes the
// vector path.  Blocks that fit on the chip at once run in one pass; more blocks run
// on resident workgroups, each group getting a share of them in proportion to its
// blocks.  Returns false (nothing launched) otherwise.
template <typename Tw, typename Tx, bool PK>
bool launch_spmv_rows(const darb_plan &p, const void *values, const uint8_t *offsets,
                      const void *offs, const void *x, float *y, const float *scales,
                      hipStream_t st, hipError_t *err) {
    constexpr int VEC = WVec<Tw>::VEC;
    // vectors per lane: up to 8 (of 4 or 8 weights)
    constexpr int KVMAX = kVmax;
    if (p.N > kLdsMaxFloats || p.M >= (int64_t(1) << 31)) return false;
    if (reinterpret_cast<uintptr_t>(x) % 16 != 0 || (p.N * int64_t(sizeof(Tx))) % 16 != 0)
        return false;
    // x rounded up to whole 1 KiB DMA chunks, then 1 KiB more: a gather at any offset
    // byte (c < N + 256) stays inside the allocation
    const size_t lds = ((size_t(p.N) * sizeof(Tx) + 1023) & ~size_t(1023)) + 1024;
    if (lds > 65536) return false;
    const int64_t cus = p.cus > 0 ? p.cus : 256;
    int64_t per_cu = kLdsPerCu / int64_t(lds);
    per_cu = per_cu > 8 ? 8 : per_cu;
    const int64_t resident = cus * per_cu;
    ProductSchedule s;
    for (int vmax = KVMAX;; vmax /= 2) {
        // a launch with fewer blocks than CUs spreads rows over more lanes
        if (!spmv_schedule<Tw>(p, values, offsets, s, vmax)) return false;
        if (vmax <= 2 || s.block_begin[s.nbins] >= cus) break;
    }
    SpmvRowsArgs a{};
    a.values = values;
    a.offs = offs;
    a.x = x;
    a.y = y;
    a.perm = p.d_perm;
    a.scales = scales;
    a.N = int32_t(p.N);
    int kv = 0;
    int64_t total = 0, blocks[kMaxBins] = {};
    for (int g = 0; g < p.bins.nbins; ++g) {
        if (s.vec[g] != VEC) return false;
        const int64_t nvec = p.bins.nblk[g] / VEC;
        const int lgL = s.log2_lanes[g];
        const int64_t rows_per_wave = int64_t(kWave) >> lgL;
        blocks[g] =
            ((p.bins.rows[g] + rows_per_wave - 1) / rows_per_wave + kSpmvWaves - 1) / kSpmvWaves;
        const int64_t n = (nvec + (int64_t(1) << lgL) - 1) >> lgL;
        if (nvec >= (int64_t(1) << 23) || n > KVMAX || blocks[g] > 0x7FFFFFFF) return false;
        a.g[g].geo = int32_t((nvec << 8) | (lgL << 3) | p.bins.log2b[g]);
        a.g[g].rows = int32_t(p.bins.rows[g]);
        a.g[g].first_row = int32_t(p.bins.first_row[g]);
        a.g[g].blocks = int32_t(blocks[g]);
        a.g[g].first_elem = p.bins.first_elem[g];
        a.g[g].first_word = p.bins.first_word[g];
        kv = n > kv ? int(n) : kv;
        total += blocks[g];
    }
    if (total == 0) return false;
    const bool loop = total > resident;
    int max_stride = 0;
    for (int g = 0; g < p.bins.nbins; ++g) {
        // resident workgroups in proportion to the group's blocks (at least one)
        int64_t sg = loop ? (blocks[g] * resident) / total : blocks[g];
        sg = sg < 1 ? 1 : (sg > blocks[g] ? blocks[g] : sg);
        a.stride[g] = int32_t(sg);
        max_stride = sg > max_stride ? int(sg) : max_stride;
    }
    const dim3 grid(unsigned(max_stride), unsigned(p.bins.nbins));
    // the kernel's unrolled vector count: the smallest of 4, 6, 8 that holds every lane's
    // vectors (fewer unrolled steps, fewer uniform branches)
#define DARB_ROWS(KV, L)                                                                    \
    hipLaunchKernelGGL((spmv_rows_kernel<Tw, Tx, KV, PK, L>), grid, dim3(kSpmvThreads), lds, st, a)
    constexpr int KV6 = KVMAX > 6 ? 6 : KVMAX;
    if (kv <= 4 || KVMAX == 4) {
        if (loop) DARB_ROWS(4, true);
        else DARB_ROWS(4, false);
    } else if (kv <= 6) {
        if (loop) DARB_ROWS(KV6, true);
        else DARB_ROWS(KV6, false);
    } else {
        if (loop) DARB_ROWS(KVMAX, true);
        else DARB_ROWS(KVMAX, false);
    }
#undef DARB_ROWS
    *err = hipGetLastError();
    return true;
}

template <typename Tw, typename Tx, bool PK>
hipError_t launch_spmv_t(const darb_plan &p, const void *values, const uint8_t *offsets,
                         const uint32_t *packed, const void *x, float *y, const float *scales,
                         hipStream_t st) {
    // Up to kVmax vectors per lane, but a launch with fewer workgroups than compute
    // units leaves CUs idle while each lane waits on a long run of loads: then rows
    // spread over more lanes (4, then 2 vectors per lane).  INT8 and fp16 vectors hold
    // 8 weights, so their small matrices need this most.
    {
        const void *offs0 = offset_source(p, offsets, packed);
        hipError_t err = hipSuccess;
        if (launch_spmv_rows<Tw, Tx, PK>(p, values, offsets, offs0, x, y, scales, st, &err))
            return err;
    }
    // otherwise (x past LDS, misaligned or scalar-path groups) the general kernel
    ProductSchedule s;
    const int64_t cus = p.cus > 0 ? p.cus : 256;
    for (int vmax = kVmax;; vmax /= 2) {
        if (!spmv_schedule<Tw>(p, values, offsets, s, vmax)) return hipErrorInvalidConfiguration;
        if (vmax <= 2 || s.block_begin[s.nbins] >= cus) break;
    }
    const int blocks = s.block_begin[s.nbins];
    if (blocks == 0) return hipSuccess;
    const Tw *v = static_cast<const Tw *>(values);
    const void *offs = offset_source(p, offsets, packed);
    const Tx *xx = static_cast<const Tx *>(x);
    const int N = int(p.N);
    // Every workgroup stages x once: launch no more of them than fit on the chip at
    // once (by LDS, at most 8 per CU) and let each take several blocks.
    const int64_t lds_per_group = p.N <= kLdsMaxFloats ? p.N * int64_t(sizeof(float)) : 0;
    int64_t per_cu = lds_per_group > 0 ? kLdsPerCu / lds_per_group : 8;
    per_cu = per_cu < 1 ? 1 : (per_cu > 8 ? 8 : per_cu);
    const int64_t resident = int64_t(p.cus > 0 ? p.cus : 256) * per_cu;

    // more blocks than fit at once: the looping form (same schedule, so the same sums)
    const int blocks_l = s.block_begin[s.nbins];
    const int grid = int(blocks_l < resident ? blocks_l : resident);
    if (p.N <= kLdsMaxFloats) {
        const size_t lds = size_t(p.N) * sizeof(float);
        const int64_t nv = p.N / (16 / int64_t(sizeof(Tx)));
        const int64_t per_thread = (nv + kSpmvThreads - 1) / kSpmvThreads;
#define DARB_SPMV_LDS(SB)                                                                    \
    do {                                                                                    \
        if (grid < blocks_l)                                                                  \
            hipLaunchKernelGGL((spmv_kernel<Tw, Tx, true, SB, PK, true>), dim3(grid),       \
                               dim3(kSpmvThreads), lds, st, v, offs, xx, y, p.d_perm, N,    \
                               p.bins, s, scales, blocks_l);                                  \
        else                                                                                \
            hipLaunchKernelGGL((spmv_kernel<Tw, Tx, true, SB, PK, false>), dim3(grid),      \
                               dim3(kSpmvThreads), lds, st, v, offs, xx, y, p.d_perm, N,    \
                               p.bins, s, scales, blocks_l);                                  \
    } while (0)
        bool direct = false;
        if constexpr (std::is_same<Tx, float>::value) {
            direct = reinterpret_cast<uintptr_t>(x) % 16 == 0;
            if (direct) DARB_SPMV_LDS(0);
        }
        if (direct) {
        } else if (per_thread <= 1) DARB_SPMV_LDS(1);
        else if (per_thread <= 2) DARB_SPMV_LDS(2);
        else if (per_thread <= 4) DARB_SPMV_LDS(4);
        else if (per_thread <= 8) DARB_SPMV_LDS(8);
        else DARB_SPMV_LDS(16);
#undef DARB_SPMV_LDS
    } else {
        if (grid < blocks_l)
            hipLaunchKernelGGL((spmv_kernel<Tw, Tx, false, 1, PK, true>), dim3(grid),
                               dim3(kSpmvThreads), 0, st, v, offs, xx, y, p.d_perm, N, p.bins, s,
                               scales, blocks_l);
        else
            hipLaunchKernelGGL((spmv_kernel<Tw, Tx, false, 1, PK, false>), dim3(grid),
                               dim3(kSpmvThreads), 0, st, v, offs, xx, y, p.d_perm, N, p.bins, s,
                               scales, blocks_l);
    }
    return hipGetLastError();
}

template <typename Tw, typename Tx>
hipError_t launch_spmv_form(const darb_plan &p, const void *values, const uint8_t *offsets,
                            const uint32_t *packed, const void *x, float *y, const float *scales,
                            hipStream_t st) {
    if (offsets)
        return launch_spmv_t<Tw, Tx, false>(p, values, offsets, nullptr, x, y, scales, st);
    return launch_spmv_t<Tw, Tx, true>(p, values, nullptr, packed, x, y, scales, st);
}

inline bool spmm_schedule(const darb_plan &p, int64_t B, int cpl, size_t wbytes,
                          const void *values, const uint8_t *offsets, ProductSchedule &s) {
    s = ProductSchedule{};
    s.nbins = p.bins.nbins;
    const int64_t lanes = (B + cpl - 1) / cpl;        // lanes needed for all columns
    const int lgL = lanes >= kWave ? 6 : ilog2_ceil(lanes);
    const int64_t slabs = (lanes + (int64_t(1) << lgL) - 1) >> lgL;
    if (slabs > 0x7FFFFFFF) return false;
    s.col_slabs = int32_t(slabs);
    const int R = kWave >> lgL;
    int64_t blocks = 0;
    for (int g = 0; g < s.nbins; ++g) {
        const int64_t nblk = p.bins.nblk[g];
        // split a row group's weights over up to 8 waves, >= ~16 weights per wave: many
        // small workgroups keep every CU's share of the gathers even
        int lgKS = ilog2_ceil((nblk + 15) / 16);
        if (lgKS > 3) lgKS = 3;
        const int KS = 1 << lgKS;
        const int rows_pb = R * (kSpmmWaves / KS);
        s.log2_lanes[g] = lgL;
        s.ksplit[g] = KS;
        // pairs load as GM-element vectors when every lane's run is aligned for it
        const int64_t GM = lgL >= 4 ? 1 : (16 >> lgL);
        s.vec[g] = (GM > 1 && nblk % GM == 0 && p.bins.first_elem[g] % GM == 0 &&
                    reinterpret_cast<uintptr_t>(values) % (GM * wbytes) == 0 &&
                    offsets_aligned(offsets, int(GM))) ? 1 : 0;
        s.block_begin[g] = int32_t(blocks);
        blocks += (p.bins.rows[g] + rows_pb - 1) / rows_pb * slabs;
        if (blocks > 0x7FFFFFFF) return false;
    }
    s.block_begin[s.nbins] = int32_t(blocks);
    return true;
}

template <typename Tw, typename Tx, int CPL, bool PK>
hipError_t launch_spmm_cpl(const darb_plan &p, const ProductSchedule &s, const Tw *v,
                           const void *offs, int64_t B, const Tx *x, int64_t ldx, float *Y,
                           int64_t ldy, const float *scales, hipStream_t st) {
    const int blocks = s.block_begin[s.nbins];
    const int N = int(p.N);
    const int lgl = s.log2_lanes[0];
    // the widths between one column and 16 bytes are chosen only for rows of more
    // than 8 lanes, so only those kernels exist
    constexpr bool kEvery = CPL == 1 || CPL * int(sizeof(Tx)) == 16;
    if (!kEvery && lgl < 4) return hipErrorInvalidConfiguration;
#define DARB_SPMM(LGL)                                                                    \
    hipLaunchKernelGGL((spmm_kernel<Tw, Tx, CPL, LGL, PK>), dim3(blocks), dim3(kSpmmThreads), \
                       0, st, v, offs, x, ldx, B, Y, ldy, p.d_perm, N, p.bins, s, scales)
    switch (lgl) {
        case 0: if constexpr (kEvery) DARB_SPMM(0); break;
        case 1: if constexpr (kEvery) DARB_SPMM(1); break;
        case 2: if constexpr (kEvery) DARB_SPMM(2); break;
        case 3: if constexpr (kEvery) DARB_SPMM(3); break;
        case 4: DARB_SPMM(4); break;
        case 5: DARB_SPMM(5); break;
        default: DARB_SPMM(6); break;
    }
#undef DARB_SPMM
    return hipGetLastError();
}

// Lanes per row of the LDS-slab SpMM (slab = 4 * lanes columns), or -1 when it does
// not apply: fp32 X, a slab of >= 32 columns whose N rows fit in LDS, and enough
// slabs (>= 128) to give every CU a workgroup.
inline int xlds_lgl(const darb_plan &p, int64_t B) {
    for (int lgl = 4; lgl >= 3; --lgl) {
        const int64_t sc = int64_t(4) << lgl;
        if (p.N * sc <= kXldsFloats && (B + sc - 1) / sc >= 128) return lgl;
    }
    return -1;
}

template <typename Tw, typename Tx, bool PK>
hipError_t launch_spmm_t(const darb_plan &p, const void *values, const uint8_t *offsets,
                         const uint32_t *packed, int64_t B, const void *X, int64_t ldx, float *Y,
                         int64_t ldy, const float *scales, hipStream_t st) {
    constexpr int CPL = 16 / int(sizeof(Tx));
    if constexpr (std::is_same<Tx, float>::value && !kScaled<Tw>) {
        // the LDS-slab kernel is chosen from the plan and B alone (rows in whole steps
        // of 16 weights, slabs that fit, enough of them), so every alignment of the
        // pointers and both offset forms take it and give the same bits; alignment
        // only chooses vector or element loads
        int lgl = xlds_lgl(p, B);
        for (int g = 0; g < p.bins.nbins; ++g)
            if (p.bins.nblk[g] % kXldsStep != 0 || p.bins.first_elem[g] % kXldsStep != 0)
                lgl = -1;
        if (lgl >= 0) {
            ProductSchedule s;
            if (!spmm_schedule(p, B, CPL, sizeof(Tw), values, offsets, s))
                return hipErrorInvalidConfiguration;
            const int64_t slabs = (B + (int64_t(4) << lgl) - 1) / (int64_t(4) << lgl);
            if (slabs > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
            const Tw *v = static_cast<const Tw *>(values);
            const float *x = static_cast<const float *>(X);
            const void *offs = offset_source(p, offsets, packed);
            const bool elem = reinterpret_cast<uintptr_t>(values) % 16 != 0 ||
                              !offsets_aligned(offsets, kXldsStep);
            const bool xvec = reinterpret_cast<uintptr_t>(X) % 16 == 0 && ldx % 4 == 0 &&
                              B % 4 == 0;
#define DARB_XLDS(LG, E)                                                                    \
    hipLaunchKernelGGL((spmm_xlds_kernel<Tw, LG, PK, E>), dim3(unsigned(slabs)),           \
                       dim3(kXldsThreads), 0, st, v, offs, x, ldx, B, Y, ldy, p.d_perm,      \
                       int(p.N), p.bins, s, xvec)
            if (lgl == 4) {
                if (elem) DARB_XLDS(4, true);
                else DARB_XLDS(4, false);
            } else {
                if (elem) DARB_XLDS(3, true);
                else DARB_XLDS(3, false);
            }
#undef DARB_XLDS
            return hipGetLastError();
        }
    }
    // columns per lane: 16 bytes of X when that leaves a row at least 5 lanes (a
    // group of 8); for smaller batches the fewest columns that keep a row within 16
    // lanes, so the launch still has many waves.  The width must divide B and keep
    // the loads aligned.  (Measured: 16-byte loads on 8 lanes beat 8-byte loads on 16;
    // rows of 2 or 4 lanes leave too few waves.)
    auto fits = [&](int c) {
        const int64_t bytes = int64_t(c) * int64_t(sizeof(Tx));
        return B % c == 0 && reinterpret_cast<uintptr_t>(X) % bytes == 0 &&
               (ldx * int64_t(sizeof(Tx))) % bytes == 0;
    };
    int cpl = 1;
    if ((B + CPL - 1) / CPL > 4 && fits(CPL)) {
        cpl = CPL;
    } else {
        while (cpl < CPL && (B + cpl - 1) / cpl > kRowLanes && fits(2 * cpl)) cpl *= 2;
    }
    ProductSchedule s;
    if (!spmm_schedule(p, B, cpl, sizeof(Tw), values, offsets, s))
        return hipErrorInvalidConfiguration;
    if (s.block_begin[s.nbins] == 0) return hipSuccess;
    const Tw *v = static_cast<const Tw *>(values);
    const void *offs = offset_source(p, offsets, packed);
    const Tx *x = static_cast<const Tx *>(X);
    if (cpl == 1)
        return launch_spmm_cpl<Tw, Tx, 1, PK>(p, s, v, offs, B, x, ldx, Y, ldy, scales, st);
    if (cpl == 2)
        return launch_spmm_cpl<Tw, Tx, 2, PK>(p, s, v, offs, B, x, ldx, Y, ldy, scales, st);
    if (cpl == 4)
        return launch_spmm_cpl<Tw, Tx, 4, PK>(p, s, v, offs, B, x, ldx, Y, ldy, scales, st);
    if constexpr (CPL == 8)
        return launch_spmm_cpl<Tw, Tx, 8, PK>(p, s, v, offs, B, x, ldx, Y, ldy, scales, st);
    return hipErrorInvalidConfiguration;
}

template <typename Tw, typename Tx>
hipError_t launch_spmm_form(const darb_plan &p, const void *values, const uint8_t *offsets,
                            const uint32_t *packed, int64_t B, const void *X, int64_t ldx,
                            float *Y, int64_t ldy, const float *scales, hipStream_t st) {
    if (offsets)
        return launch_spmm_t<Tw, Tx, false>(p, values, offsets, nullptr, B, X, ldx, Y, ldy,
                                            scales, st);
    return launch_spmm_t<Tw, Tx, true>(p, values, nullptr, packed, B, X, ldx, Y, ldy, scales,
                                       st);
}

}  // namespace
}  // namespace darb
