// Device-side readers of the bit-packed offsets, shared by the products and the
// unpack kernel.
//
// Section 4.2 stores the position of a block's kept weight in log2 b bits.  The
// packed form used here: inside one block-size group (log2 b = l) the retained
// weights are numbered j = 0, 1, ... in storage order and cut into runs of 32;
// run j / 32 is l consecutive 32-bit words, and weight j's index is bits
// (j % 32) * l ... (j % 32) * l + l - 1 of its run read as one little-endian bit
// string.  Groups follow each other in ascending block size; a group with l = 0
// (b = 1: every index is 0) has no words.  A run never straddles a group, so any
// slice of consecutive weights that starts at a multiple of 4, 8 or 16 inside
// its group lies inside one run.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace darb {

// The packed offsets of one group.  `words` must be a readable device address
// even for l = 0 (the readers then load one word and mask it to nothing).
struct PackedGroup {
    const uint32_t *words;   // the group's first word
    int l;                   // log2 b
    int lc;                  // max(l, 1): words a run spans, for index clamping
    uint32_t mask;           // (1 << l) - 1
};

__device__ __forceinline__ PackedGroup packed_group(const uint32_t *words, int64_t first_word,
                                                    int l) {
    return PackedGroup{words + first_word, l, l > 0 ? l : 1, (1u << l) - 1u};
}

// The words holding group weights j, j + 1, ... and where they start.  Word
// indices are clamped into the run: bits past the run's end are never an index
// of this run, and callers only use bits of weights inside it.
struct PackedWords2 { uint32_t a, b; int sh; };
struct PackedWords3 { uint32_t a, b, c; int sh; };

__device__ __forceinline__ PackedWords2 packed_load2(const PackedGroup &pg, int64_t j) {
    const uint32_t *run = pg.words + (j >> 5) * pg.l;
    const int bit = int(j & 31) * pg.l;
    const int w = bit >> 5;
    return PackedWords2{run[w], run[w + 1 < pg.lc ? w + 1 : pg.lc - 1], bit & 31};
}

__device__ __forceinline__ PackedWords3 packed_load3(const PackedGroup &pg, int64_t j) {
    const uint32_t *run = pg.words + (j >> 5) * pg.l;
    const int bit = int(j & 31) * pg.l;
    const int w = bit >> 5;
    return PackedWords3{run[w], run[w + 1 < pg.lc ? w + 1 : pg.lc - 1],
                        run[w + 2 < pg.lc ? w + 2 : pg.lc - 1], bit & 31};
}

// 32 bits starting at weight j's first bit (enough for 4 indices of <= 7 bits).
__device__ __forceinline__ uint32_t packed_bits32(const PackedWords2 &p) {
    return uint32_t(((uint64_t(p.b) << 32) | p.a) >> p.sh);
}

// 64 bits starting at weight j's first bit (enough for 8 indices of <= 7 bits).
__device__ __forceinline__ uint64_t packed_bits64(const PackedWords3 &p) {
    const uint64_t lo = ((uint64_t(p.b) << 32) | p.a) >> p.sh;
    return p.sh ? lo | (uint64_t(p.c) << (64 - p.sh)) : lo;
}

// Index q of a bit string that starts at an index boundary.
template <typename Bits>
__device__ __forceinline__ int packed_field(Bits bits, int q, const PackedGroup &pg) {
    return int(uint32_t(bits >> (q * pg.l)) & pg.mask);
}

}  // namespace darb
