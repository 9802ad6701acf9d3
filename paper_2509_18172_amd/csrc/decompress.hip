// SBVR -> binary16 decompression, the prefill path: the decoded matrix
// W[o][128 g + j] = sum_i c[o][g][i] b[o][g][i][j] (Sec. 4.1) is written as
// binary16 so that a dense matrix-core GEMM can consume it.  A sum of at most
// four binary16 values is exact in binary64 (53-bit significand), so rounding
// it once to binary16 (to nearest, ties to even) gives the correctly rounded
// weight -- the same as rounding the exact decoded value.
//
// Workgroup = one (tile, gblock) block of the device format: TR rows x 512
// columns.  Each of its TR x 4 (row, group) pairs has 2^k distinct decoded
// values (the subset sums); the workgroup rounds them once into an LDS table
// (one entry per thread), then thread = 8 consecutive columns of one row
// gathers its k plane words (the device bit layout puts element 8v+p of a
// word at bit 4p+v, so (w >> v) & 0x11111111 holds its 8 bits in nibbles
// 0..7), forms the 4-bit subset index of each element and looks it up, and
// writes 16 bytes.  HBM-bound: per weight it reads k/8 + 2k/128 bytes and
// writes 2.
#include "device_ops.h"
#include "f16_round.h"
#include "launch.h"

namespace sbvr {

// One workgroup per (tile, gblock) block; the plane words are loaded first so
// that their latency overlaps the subset-sum table.  (Several blocks per
// workgroup in a software pipeline measured slower.)
// IX: coefficient-cache format -- coeffs is then the device index blocks and
// the coefficients come from table (n_sets sets of TABLE_STRIDE entries; an
// index past the end gives zero coefficients).
template <int K, bool IX>
__global__ void __launch_bounds__(1024) decompress_kernel(Dims d, const uint32_t *__restrict__ planes,
                                                          const uint16_t *__restrict__ coeffs,
                                                          const uint16_t *__restrict__ table, int n_sets,
                                                          uint16_t *__restrict__ W)
{
    constexpr int TR = tile_rows(K), NSUB = 1 << K;
    __shared__ uint16_t lut[TR * GB * NSUB];  // [row][group slot][subset]
    const size_t blk = blockIdx.x;
    const int tile = (int)(blk / d.n_gblocks), gb = (int)(blk % d.n_gblocks);
    const int t = threadIdx.x;
    const int r = t >> 6, c8 = t & 63;  // row in the tile, 8-column chunk in the gblock
    const int b = c8 >> 4;               // group slot
    const int wq = (c8 & 15) >> 2;       // word of the group
    const int v = c8 & 3;                // elements 8v .. 8v+7 of the word
    const int o = tile * TR + r, g = gb * GB + b;
    // plane words first (padding rows and groups of the block are zero)
    const uint32_t *pw = planes + blk * plane_block_words(K) + (size_t)((b * TR + r) * K) * 4 + wq;
    uint32_t w[K];
#pragma unroll
    for (int i = 0; i < K; ++i)
        w[i] = pw[i * 4];

    const uint16_t *cb = coeffs + blk * (IX ? index_block_entries(K) : coeff_block_entries(K));
    for (int e = t; e < TR * GB * NSUB; e += blockDim.x) {
        const int sub = e % NSUB, rb = e / NSUB, lb = rb % GB, lr = rb / GB;
        int set = 0;
        if constexpr (IX)
            set = cb[index_entry(K, lr, lb)];
        double s = 0.0;  // exact: at most K binary16 terms
#pragma unroll
        for (int i = 0; i < K; ++i) {
            if (!((sub >> i) & 1))
                continue;
            uint16_t c;
            if constexpr (IX)
                c = set < n_sets ? table[(size_t)set * TABLE_STRIDE + i] : (uint16_t)0;
            else
                c = cb[coeff_entry(K, lr, lb, i)];
            s += (double)half_bits_to_float(c);
        }
        lut[e] = f64_to_f16_rne(s);
    }
    __syncthreads();
    if (o >= d.O || g >= d.G)
        return;
    uint32_t sub = 0;  // nibble p: subset index of element 8v+p
#pragma unroll
    for (int i = 0; i < K; ++i)
        sub |= ((w[i] >> v) & 0x11111111u) << i;
    const uint16_t *L = lut + (r * GB + b) * NSUB;
    uint32_t out[4];
#pragma unroll
    for (int h = 0; h < 4; ++h)
        out[h] = (uint32_t)L[(sub >> (8 * h)) & 0xf] | ((uint32_t)L[(sub >> (8 * h + 4)) & 0xf] << 16);
    *(uint4 *)(W + (size_t)o * d.I + (size_t)g * GROUP + wq * 32 + 8 * v) = make_uint4(out[0], out[1], out[2], out[3]);
}

template <bool IX>
static const void *decompress_kernel_for(int k)
{
    return k == 4   ? (const void *)decompress_kernel<4, IX>
           : k == 3 ? (const void *)decompress_kernel<3, IX>
           : k == 2 ? (const void *)decompress_kernel<2, IX>
                    : (const void *)decompress_kernel<1, IX>;
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
    const void *fn = ix ? decompress_kernel_for<true>(d.k) : decompress_kernel_for<false>(d.k);
    const unsigned grid = (unsigned)((size_t)d.n_tiles * d.n_gblocks);
    return launch_kernel(fn, dim3(grid), dim3(64 * d.tr), 0, stream, args);
}

}  // namespace sbvr
