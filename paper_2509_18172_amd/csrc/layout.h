// Device layout of SBVR weights for the gfx950 GEMV kernels.
//
// The canonical format (include/sbvr.h) stores, per (row o, group g, plane i),
// 128 plane bits in four 32-bit words plus one binary16 coefficient
// (Sec. 4.1, Sec. 4.4).  The device format regroups those words so that a
// wavefront's 128-bit loads are contiguous and so that each loaded word can be
// turned into matrix-core operands with a handful of bit masks.
//
// A matrix-core instruction has 16 A rows; they hold (tile row r, plane i)
// pairs, m = r * RS + i, with RS = 16 / TR "row slots" per tile row:
//
//   k     tile rows TR   row slots RS   rows used
//   1          16             1            16
//   2           8             2            16
//   3           4             4            12 (plane slot 3 stays empty)
//   4           4             4            16
//
//   gblock    GB = 4 consecutive groups (512 inner-dimension elements)
//   block     one (tile, gblock) pair; blocks are stored tile-major:
//             block index = tile * n_gblocks + gblock
//
//   plane block (GB * TR * k * 16 bytes): slot (b * TR + r) * k + i holds the
//     four words (16 bytes) of plane i of row TR*tile + r for group
//     4*gblock + b -- 1 KiB for k = 1, 2, 4.
//   coeff block (GB * TR * k * 2 bytes): the coefficient of A row m = 4q + j
//     (= tile row r, plane i) of group slot b is entry (q * GB + b) * CPL + j,
//     CPL = 4 (3 for k = 3, whose rows m = 4r + i have i < 3).  A lane of a
//     16x16 result holds rows 4q .. 4q+3: their coefficients are contiguous
//     for one group slot (CPL entries) and for all four (4 * CPL entries).
//
// Within each device word the bits are transposed as a 4 x 8 bit matrix:
// element e = 8 v + p (0 <= v < 4, 0 <= p < 8) of the word sits at bit 4 p + v.
// Then w & (0x11111111 << v) places element 8 v + p in nibble p, which is the
// matrix-core k-slot 8 v + p of an fp4 operand register v.
//
// Rows past O and groups past G are zero padding (zero planes and zero
// coefficients contribute nothing to y).
#pragma once

#include <stddef.h>
#include <stdint.h>

#define SBVR_HD __host__ __device__ __forceinline__

namespace sbvr {

constexpr int GROUP = 128;     // weights per SBVR group (Sec. 4.1)
constexpr int GB = 4;          // groups per gblock
constexpr int MAX_K = 4;       // planes supported by this build

// rows per tile and A-row slots per tile row for k planes
SBVR_HD constexpr int tile_rows(int k) { return k == 1 ? 16 : (k == 2 ? 8 : 4); }
SBVR_HD constexpr int row_slots(int k) { return 16 / tile_rows(k); }

struct Dims {
    int O, I, k, G, tr, n_tiles, n_gblocks;
};

SBVR_HD Dims make_dims(int O, int I, int k)
{
    Dims d;
    d.O = O;
    d.I = I;
    d.k = k;
    d.G = I / GROUP;
    d.tr = tile_rows(k);
    d.n_tiles = (O + d.tr - 1) / d.tr;
    d.n_gblocks = (d.G + GB - 1) / GB;
    return d;
}

SBVR_HD constexpr int coefs_per_quad(int k) { return k == 3 ? 3 : 4; }

// coefficient entry of (tile row r, group slot b, plane i) within a block
SBVR_HD int coeff_entry(int k, int r, int b, int i)
{
    const int m = r * row_slots(k) + i;
    return ((m / 4) * GB + b) * coefs_per_quad(k) + m % 4;
}

SBVR_HD size_t plane_block_words(int k) { return (size_t)GB * tile_rows(k) * k * 4; }
SBVR_HD size_t coeff_block_entries(int k) { return (size_t)GB * tile_rows(k) * k; }

SBVR_HD size_t plane_bytes(const Dims &d)
{
    return (size_t)d.n_tiles * d.n_gblocks * plane_block_words(d.k) * 4;
}

SBVR_HD size_t coeff_bytes(const Dims &d)
{
    return (size_t)d.n_tiles * d.n_gblocks * coeff_block_entries(d.k) * 2;
}

// Coefficient-cache format (Sec. 4.4): one 16-bit coefficient-set index per
// (row, group) instead of k coefficients.  Index block of a (tile, gblock)
// block: GB * TR entries; the entry of (tile row r, group slot b) is
// ((r / NP) * GB + b) * NP + r % NP with NP = TR / 4, so the lane that holds
// the result rows of tile rows NP*q .. NP*q+NP-1 for group slot b finds their
// indices in NP consecutive entries.  The cache itself (the table of
// coefficient sets) is stored with TABLE_STRIDE entries per set, zero padded.
constexpr int TABLE_STRIDE = 4;
constexpr int MAX_SETS = 65536;  // 16-bit index

SBVR_HD constexpr int index_per_lane(int k) { return tile_rows(k) / 4; }

SBVR_HD int index_entry(int k, int r, int b)
{
    const int np = index_per_lane(k);
    return ((r / np) * GB + b) * np + r % np;
}

SBVR_HD size_t index_block_entries(int k) { return (size_t)GB * tile_rows(k); }

SBVR_HD size_t index_bytes(const Dims &d)
{
    return (size_t)d.n_tiles * d.n_gblocks * index_block_entries(d.k) * 2;
}

SBVR_HD size_t table_bytes(int n_sets) { return (size_t)n_sets * TABLE_STRIDE * 2; }

// canonical bit t (element t of the word) -> device bit position
SBVR_HD int device_bit_of(int t) { return 4 * (t % 8) + t / 8; }
// device bit position d -> canonical bit (element index within the word)
SBVR_HD int canonical_bit_of(int d) { return 8 * (d % 4) + d / 4; }

SBVR_HD uint32_t to_device_word(uint32_t w)
{
    uint32_t r = 0;
    for (int t = 0; t < 32; ++t)
        r |= ((w >> t) & 1u) << device_bit_of(t);
    return r;
}

SBVR_HD uint32_t to_canonical_word(uint32_t w)
{
    uint32_t r = 0;
    for (int d = 0; d < 32; ++d)
        r |= ((w >> d) & 1u) << canonical_bit_of(d);
    return r;
}

}  // namespace sbvr
