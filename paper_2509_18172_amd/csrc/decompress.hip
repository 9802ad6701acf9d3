// SBVR -> binary16 decompression, the prefill path: the decoded matrix
// W[o][128 g + j] = sum_i c[o][g][i] b[o][g][i][j] (Sec. 4.1) is written as
// binary16 so that a dense matrix-core GEMM can consume it.  A sum of at most
// four binary16 values is exact in binary64 (53-bit significand), so rounding
// it once to binary16 (to nearest, ties to even) gives the correctly rounded
// weight -- the same as rounding the exact decoded value.  When the
// coefficients' exponents span at most 11 the sum is exact in binary32 as
// well and the hardware conversion rounds it (the common case; binary64
// otherwise).
//
// A (tile, gblock) block of the device format is TR rows x 512 columns.  Each
// of its TR x 4 (row, group) pairs has 2^k distinct decoded values (the subset
// sums), rounded once into an LDS table; then a lane = 8 consecutive columns
// of one row takes its k plane words (the device bit layout puts element 8v+p
// of a word at bit 4p+v, so (w >> v) & 0x11111111 holds its 8 bits in nibbles
// 0..7), forms the subset index of each element, looks it up and writes 16
// bytes.  HBM-bound: per weight it reads k/8 + 2k/128 bytes and writes 2.
#include "device_ops.h"
#include "lds_lookup.h"
#include "f16_round.h"
#include "launch.h"

namespace sbvr {

// Broadcast within each quad of lanes: every lane gets lane i's value.
__device__ __forceinline__ uint32_t quad_bcast(uint32_t v, int i)
{
    switch (i) {
    case 0:
        return __builtin_amdgcn_update_dpp(0u, v, 0x00, 0xf, 0xf, false);  // quad_perm [0,0,0,0]
    case 1:
        return __builtin_amdgcn_update_dpp(0u, v, 0x55, 0xf, 0xf, false);  // [1,1,1,1]
    case 2:
        return __builtin_amdgcn_update_dpp(0u, v, 0xaa, 0xf, 0xf, false);  // [2,2,2,2]
    default:
        return __builtin_amdgcn_update_dpp(0u, v, 0xff, 0xf, 0xf, false);  // [3,3,3,3]
    }
}

// A workgroup decodes NB consecutive gblocks of one tile; wavefront r of the
// workgroup is row r of the tile.
//   * Plane words: lane (slot b, word wq, v) loads word wq of plane v, so a
//     group slot's 16 lanes read its 64 contiguous bytes with one load, and
//     the quad (b, wq) then holds word wq of every plane; each lane takes all
//     k of them from its quad by DPP broadcasts.
//   * Table: wavefront r builds the 4 x 2^k entries of its own row (lane l:
//     slot l / 2^k, subset l % 2^k) from the row's coefficients, read as one
//     contiguous run per slot.  Only that wavefront reads them back, so no
//     workgroup barrier is needed: one wavefront's LDS operations complete in
//     order.
//   * Output: 16 bytes per lane and gblock, stored non-temporally (the matrix
//     is written once and read later by the GEMM).
// IX: coefficient-cache format -- coeffs is then the device index blocks and
// the coefficients come from table (n_sets sets of TABLE_STRIDE entries; an
// index past the end gives zero coefficients).
template <int K, bool IX, int NB>
__global__ void __launch_bounds__(1024) decompress_kernel(Dims d, const uint32_t *__restrict__ planes,
                                                          const uint16_t *__restrict__ coeffs,
                                                          const uint16_t *__restrict__ table, int n_sets,
                                                          uint16_t *__restrict__ W)
{
    constexpr int TR = tile_rows(K), NSUB = 1 << K, NE = TR * GB * NSUB, ROW_E = GB * NSUB;
    __shared__ uint16_t lut[NB][NE];  // [gblock][row][group slot][subset]
    const int gpt = (d.n_gblocks + NB - 1) / NB;
    const int tile = (int)(blockIdx.x / gpt), gb0 = (int)(blockIdx.x % gpt) * NB;
    const int r = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int b = lane >> 4;         // group slot
    const int wq = (lane & 15) >> 2; // word of the group
    const int v = lane & 3;          // elements 8v .. 8v+7 of the word; plane v for the load
    const int o = tile * TR + r;
    const size_t blk0 = (size_t)tile * d.n_gblocks + gb0;

    // plane words first, so that their latency overlaps the table
    uint32_t mine[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
        const bool ok = gb0 + u < d.n_gblocks && v < K;
        mine[u] = ok ? planes[(blk0 + u) * plane_block_words(K) + (size_t)((b * TR + r) * K + v) * 4 + wq] : 0u;
    }

    for (int e2 = lane; e2 < NB * ROW_E; e2 += 64) {
        const int u = e2 / ROW_E, lb = (e2 % ROW_E) / NSUB, sub = e2 % NSUB;
        if (gb0 + u >= d.n_gblocks)
            continue;
        const uint16_t *cb = coeffs + (blk0 + u) * (IX ? index_block_entries(K) : coeff_block_entries(K));
        uint16_t c[K];
        if constexpr (IX) {
            const int set = cb[index_entry(K, r, lb)];
            const bool in = set < n_sets;
#pragma unroll
            for (int i = 0; i < K; ++i)
                c[i] = in ? table[(size_t)set * TABLE_STRIDE + i] : (uint16_t)0;
        } else {
            const uint16_t *cp = cb + coeff_entry(K, r, lb, 0);  // the row's K entries are contiguous
            if constexpr (K == 4) {
                const uint2 q = *(const uint2 *)cp;  // 8-byte aligned: entry (r * GB + lb) * 4
                c[0] = (uint16_t)(q.x & 0xffffu);
                c[1] = (uint16_t)(q.x >> 16);
                c[2] = (uint16_t)(q.y & 0xffffu);
                c[3] = (uint16_t)(q.y >> 16);
            } else {
#pragma unroll
                for (int i = 0; i < K; ++i)
                    c[i] = cp[i];
            }
        }
        uint32_t cw[K];
#pragma unroll
        for (int i = 0; i < K; ++i)
            cw[i] = c[i];
        const bool exact32 = f16_sums_exact_in_f32<K>(cw);
        uint16_t val;
        if (__builtin_amdgcn_ballot_w64(!exact32) == 0 || exact32) {
            // binary32: the sum is exact, one hardware rounding to binary16
            float s = 0.f;
#pragma unroll
            for (int i = 0; i < K; ++i)
                s += ((sub >> i) & 1) ? half_bits_to_float(c[i]) : 0.f;
            val = __half_as_ushort(__float2half_rn(s));
        } else {
            double s = 0.0;  // exact: at most K binary16 terms
#pragma unroll
            for (int i = 0; i < K; ++i)
                s += ((sub >> i) & 1) ? (double)half_bits_to_float(c[i]) : 0.0;
            val = f64_to_f16_rne(s);
        }
        lut[u][r * ROW_E + lb * NSUB + sub] = val;
    }

    uint32_t w[NB][K];
#pragma unroll
    for (int u = 0; u < NB; ++u)
#pragma unroll
        for (int i = 0; i < K; ++i)
            w[u][i] = quad_bcast(mine[u], i);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    typedef unsigned v4u_t __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int u = 0; u < NB; ++u) {
        const int g = (gb0 + u) * GB + b;
        if (o >= d.O || g >= d.G || gb0 + u >= d.n_gblocks)
            continue;
        uint32_t sub = 0;  // nibble p: subset index of element 8v+p
#pragma unroll
        for (int i = 0; i < K; ++i)
            sub |= ((w[u][i] >> v) & 0x11111111u) << i;
        const uint16_t *L = lut[u] + r * ROW_E + b * NSUB;
        // byte h of e2 / o2: byte offset of nibble 2h / 2h+1's entry; one
        // byte-select add per lookup address
        const uint32_t e2 = (sub & 0x0F0F0F0Fu) << 1, o2 = (sub >> 3) & 0x1E1E1E1Eu, Lb = lds_addr(L);
        const uint32_t a[8] = {add_byte<0>(Lb, e2), add_byte<0>(Lb, o2), add_byte<1>(Lb, e2), add_byte<1>(Lb, o2),
                               add_byte<2>(Lb, e2), add_byte<2>(Lb, o2), add_byte<3>(Lb, e2), add_byte<3>(Lb, o2)};
        auto at = [&](int i) { return (uint32_t)*(const __attribute__((address_space(3))) uint16_t *)(uintptr_t)a[i]; };
        v4u_t out;
#pragma unroll
        for (int h = 0; h < 4; ++h)
            out[h] = at(2 * h) | (at(2 * h + 1) << 16);
        __builtin_nontemporal_store(out, (v4u_t *)(W + (size_t)o * d.I + (size_t)g * GROUP + wq * 32 + 8 * v));
    }
}

// gblocks per workgroup: one for small matrices (enough workgroups to fill
// the chip), more for large ones (more bytes in flight per wavefront).
// Measured on the 8B shapes: k/v 1, q/o 2, gate/up/down 4 were fastest.
static int decompress_nb(const Dims &d)
{
    const size_t blocks = (size_t)d.n_tiles * d.n_gblocks;
    return blocks >= 16384 ? 4 : (blocks >= 4096 ? 2 : 1);
}

template <bool IX, int NB>
static const void *decompress_kernel_for(int k)
{
    return k == 4   ? (const void *)decompress_kernel<4, IX, NB>
           : k == 3 ? (const void *)decompress_kernel<3, IX, NB>
           : k == 2 ? (const void *)decompress_kernel<2, IX, NB>
                    : (const void *)decompress_kernel<1, IX, NB>;
}

template <bool IX>
static const void *decompress_kernel_for(int k, int nb)
{
    return nb == 4 ? decompress_kernel_for<IX, 4>(k)
                   : (nb == 2 ? decompress_kernel_for<IX, 2>(k) : decompress_kernel_for<IX, 1>(k));
}

int launch_decompress(const Dims &d, const WeightRef &w, uint16_t *W, hipStream_t stream)
{
    Dims dd = d;
    const uint32_t *p = (const uint32_t *)w.planes;
    const bool ix = w.index != nullptr;
    const uint16_t *c = (const uint16_t *)(ix ? w.index : w.coeffs);
    const uint16_t *t = (const uint16_t *)w.table;
    int n_sets = w.n_sets;
    void *args[] = {&dd, &p, &c, &t, &n_sets, &W};
    const int nb = decompress_nb(d);
    const void *fn = ix ? decompress_kernel_for<true>(d.k, nb) : decompress_kernel_for<false>(d.k, nb);
    const unsigned grid = (unsigned)((size_t)d.n_tiles * ((d.n_gblocks + nb - 1) / nb));
    return launch_kernel(fn, dim3(grid), dim3(64 * d.tr), 0, stream, args);
}

}  // namespace sbvr
