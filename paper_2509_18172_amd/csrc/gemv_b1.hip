// Batch-1 SBVR GEMV (Sec. 4.4): y[o] = sum_g sum_i c[o][g][i] * S[o][g][i].
//
// One-shot kernel, for matrices whose loads can all be in flight at once.
// A workgroup owns T tiles (T * TR consecutive rows, TR = 16 / row slots: 4
// rows at k = 3, 4, 8 at k = 2, 16 at k = 1); its wavefront w owns gblock
// w (512 inner elements; at most 16 per row: split-K inside the workgroup).
// Partial row sums are reduced across wavefronts in LDS in a fixed order:
// results are deterministic and there is no global workspace.  Larger
// matrices go to the streaming kernel.
//
// Block-diagonal activation operand.  One 16x16x128 instruction takes, in its
// four 32-slot k-blocks, word q of four different groups (the four groups of a
// gblock), and the 16 output columns are (group slot s, limb l): column 4s+l
// holds limb l (of four) of group s's activations in k-block s and zeros
// elsewhere.
// Four chained instructions (q = 0..3) therefore leave in D[row][4s+l] the
// complete per-plane sum of group s for limb l, and the coefficients are
// applied once per four instructions: D rows are (tile row, plane), so a lane
// multiplies its four D values by their coefficients, which belong to one
// group and to 1, 2 or 4 tile rows (k = 3..4, 2, 1).
//
// Latency hiding.  Every load a wavefront needs -- its 1 KiB of activations,
// then the T tiles' plane and coefficient blocks -- is issued before any
// arithmetic, and scheduling barriers keep the compiler from sinking weight
// loads below the activation work (left alone it does, to save registers,
// which serialises DRAM latency behind arithmetic).
#include <climits>

#include "device_ops.h"
#include "launch.h"

namespace sbvr {

// per wavefront: [q][s][l][32 B] limb chunks, then 256 zero bytes (the
// operand halves a lane does not cover read 16 of them, a different 16 for
// each lane of a 16-lane group: reading one shared chunk from most lanes
// serialised the LDS reads, about 0.3 us on the latency-bound launches)
constexpr int B1_WAVE_LDS = 2048 + 256;

template <int K, int T>
struct B1Regs {
    uint4 p[T];  // plane words of each tile (this lane's 16 bytes)
    uint2 c[T];  // the coefficients of this lane's four D rows, each tile
    typename IxLane<K>::type ix[T];  // coefficient-cache format: their set indices
    uint4 x;     // this lane's 8 activations
};

// A8: activations converted online to SBVR-8.  IX: coefficient-cache format
// (index blocks + table of coefficient sets) instead of per-group coefficients.
// The fields every wavefront needs (its first loads' addresses and sizes, and
// the output) come again as leading scalar arguments: the compiler preloads
// those into SGPRs at launch (built with -amdgpu-kernarg-preload-count), so
// neither the first loads nor the LDS waits before the matrix-core work sit
// behind a kernel-argument fetch (a scalar load shares the LDS wait counter);
// the rest are read from the struct.  The wavefront count is the gblock count.
// The kernel body for workgroup `bid` of the matrix in `a`.
template <int K, int T, bool A8, bool IX>
__device__ __forceinline__ void gemv_b1_body(const GemvArgs &a, unsigned bid)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63;
    const int wv = wave_id();
    const int nw = a.n_gblocks;  // one wavefront per gblock
    unsigned char *lds = smem + wv * B1_WAVE_LDS;
    float *red = (float *)(smem + nw * B1_WAVE_LDS);

    const int tile0 = bid * T;
    const int gb = wv;

    constexpr int TR = tile_rows(K), NP = partials_per_lane<K>();
    // A operand: row m = lane%16 = (tile row, plane), k-block = group slot;
    // lanes of empty plane slots (K = 3) read a valid slot and zero it.
    bool a_ok;
    const unsigned a_off = a_slot_bytes<K>(lane, a_ok) / 16;
    // coefficients of the lane's D rows (group slot (lane%16)/4)
    const unsigned c_off = (unsigned)(((lane >> 4) * GB + ((lane & 15) >> 2)) * coefs_per_lane<K>());
    constexpr int PBLK = GB * TR * K;  // uint4 per plane block
    constexpr int CBLK = GB * TR * K;  // coefficients per block
    // Tiles past the end (last workgroup) re-read the last tile; their rows
    // are >= O and never stored.  Block indices are wavefront-uniform, so each
    // load is a scalar base plus the lane's 32-bit offset.
    int tblk[T];
#pragma unroll
    for (int t = 0; t < T; ++t)
        tblk[t] = min(tile0 + t, a.n_tiles - 1) * a.n_gblocks;

    // coefficient-cache format: index blocks and the table, through
    // descriptors (the table's bounds the set count)
    constexpr unsigned IBLK_B = GB * TR * 2;
    const unsigned i_lane = (unsigned)(((lane >> 4) * GB + ((lane & 15) >> 2)) * index_per_lane(K)) * 2u;
    buf_rsrc irs, trs;
    if constexpr (IX) {
        irs = make_rsrc(a.index, (unsigned)((size_t)a.n_tiles * a.n_gblocks * IBLK_B));
        trs = make_rsrc(a.table, (unsigned)a.n_sets * (TABLE_STRIDE * 2));
    }

    auto fetch = [&](B1Regs<K, T> &R) {
        // activations first; lanes past I (ragged end) read a valid address
        // and are zeroed before use
        R.x = *(const uint4 *)(a.x + min(gb * (GB * GROUP) + lane * 8, a.I - 8));
        __builtin_amdgcn_sched_barrier(0);  // the operand build waits only for x
        if constexpr (IX) {  // set indices before the planes: their gathers wait only for them
#pragma unroll
            for (int t = 0; t < T; ++t)
                R.ix[t] = buf_index<K>(irs, (unsigned)(tblk[t] + gb) * IBLK_B + i_lane);
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const size_t blk = (size_t)(tblk[t] + gb);
            const uint4 v = load_nt16(a.planes + blk * PBLK + a_off);
            R.p[t] = a_ok ? v : make_uint4(0u, 0u, 0u, 0u);
            if constexpr (!IX)
                R.c[t] = load_coefs4<K>(a.coeffs + blk * CBLK + c_off);
        }
    };

    // limb writes: lane owns elements 8*lane .. 8*lane+7 of the gblock:
    // group slot lane/16, word (lane%16)/4, k-slots 8*(lane%4) ..
    const int wr_off = ((((lane & 15) >> 2) * 4 + (lane >> 4)) * 4) * 32 + 8 * (lane & 3);
    // B-operand reads: column n = lane%16 = (slot s, limb l), k-block lane/16.
    // fp8 k-blocks: registers 0-3 hold k = 16 kb + [0,16), registers 4-7 hold
    // k = 64 + 16 kb + [0,16); slot s covers k = 32 s + [0,32).
    const int n = lane & 15, kb = lane >> 4;
    const int s = n >> 2, l = n & 3;
    // limbs 2 and 3 of the SBVR-8 codes are zero: those columns read zeros
    const bool act = (!A8 || l < 2) && ((kb >> 1) == (s & 1));
    const int data_off = (s * 4 + l) * 32 + 16 * (kb & 1);
    const int zero_off = 2048 + 16 * (lane & 15);
    // the k-block half a lane does not cover reads the zero chunk for every q
    const int lo_off = (act && s < 2) ? data_off : zero_off;
    const int hi_off = (act && s >= 2) ? data_off : zero_off;
    const int lo_step = (act && s < 2) ? 512 : 0;
    const int hi_step = (act && s >= 2) ? 512 : 0;
    const int inv_alpha = inv_alpha_exp(lane & 3);

    float acc[T][NP];
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
        for (int p = 0; p < NP; ++p)
            acc[t][p] = 0.f;

    // Activation limbs of the gblock in R -> LDS -> the four B operands;
    // returns the factor that undoes the activation scaling (2^-sigma; with
    // SBVR-8 activations the lane's group scale).
    auto operands = [&](const B1Regs<K, T> &R, v8i *Bq) -> float {
        const uint4 xv = gb * (GB * GROUP) + lane * 8 < a.I ? R.x : make_uint4(0u, 0u, 0u, 0u);
        float out_scale;
        Limbs L;
        if constexpr (A8) {
            L = a8_limbs(xv, lane, inv_alpha, out_scale);
        } else {
            const int sigma = scale_exponent(wave_absmax_h(xv));
            L = split_limbs(xv, sigma, inv_alpha);
            out_scale = ldexpf(1.0f, -sigma);
        }
        // same wavefront: the LDS writes complete before the reads below
#pragma unroll
        for (int j = 0; j < (A8 ? 2 : 4); ++j)
            *(uint2 *)(lds + wr_off + j * 32) = make_uint2(L.l[j][0], L.l[j][1]);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            Bq[q] = lds_operand(lds + lo_off + q * lo_step, lds + hi_off + q * hi_step);
        return out_scale;
    };
    // The T tiles of the gblock in R.
    auto tiles = [&](const B1Regs<K, T> &R, const v8i *Bq, float inv_scale) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
            v4f d = {0.f, 0.f, 0.f, 0.f};
            d = mfma_fp4_fp8<A8>(fp4_operand(R.p[t].x), Bq[0], d);
            d = mfma_fp4_fp8<A8>(fp4_operand(R.p[t].y), Bq[1], d);
            d = mfma_fp4_fp8<A8>(fp4_operand(R.p[t].z), Bq[2], d);
            d = mfma_fp4_fp8<A8>(fp4_operand(R.p[t].w), Bq[3], d);
            float part[NP];
            apply_coefs<K>(R.c[t], d, part);
#pragma unroll
            for (int p = 0; p < NP; ++p)
                acc[t][p] = fmaf(part[p], inv_scale, acc[t][p]);
        }
    };

    // the zero region read by the columns of the other k-blocks
    *(uint32_t *)(lds + 2048 + 4 * lane) = 0u;

    {
        B1Regs<K, T> R;
        fetch(R);
        __builtin_amdgcn_sched_barrier(0);  // all loads issued before arithmetic
        if constexpr (IX) {  // coefficient sets, gathered while the operands are built
#pragma unroll
            for (int t = 0; t < T; ++t)
                R.c[t] = table_coefs4<K>(trs, R.ix[t]);
            __builtin_amdgcn_sched_barrier(0);
        }
        v8i Bq[4];
        const float inv_scale = operands(R, Bq);
        __builtin_amdgcn_sched_barrier(0);
        tiles(R, Bq, inv_scale);
    }

    // sum the 16 columns (group slot x limb) of each row ...
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
        for (int p = 0; p < NP; ++p)
            acc[t][p] = row16_sum(acc[t][p]);
    const int row_base = tile0 * TR;
    // lane rows: (lane / 16) * NP + p within the tile
    const int lrow = (lane >> 4) * NP;
    if (nw == 1) {  // inner dimension not split: store directly
        if ((lane & 15) == 0) {
#pragma unroll
            for (int t = 0; t < T; ++t)
#pragma unroll
                for (int p = 0; p < NP; ++p) {
                    const int o = row_base + t * TR + lrow + p;
                    if (o < a.O)
                        a.y[o] = __half_as_ushort(__float2half_rn(acc[t][p]));
                }
        }
        return;
    }
    // ... then the wavefronts, in wavefront order
    if ((lane & 15) == 0) {
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int p = 0; p < NP; ++p)
                red[(wv * T + t) * TR + lrow + p] = acc[t][p];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < T * TR; idx += 64 * nw) {
        const int o = row_base + idx;
        if (o < a.O) {
            float v = 0.f;
            for (int w = 0; w < nw; ++w)
                v += red[w * T * TR + idx];
            a.y[o] = __half_as_ushort(__float2half_rn(v));
        }
    }
}

template <int K, int T, bool A8, bool IX>
__global__ void __launch_bounds__(1024) gemv_b1_kernel(const uint4 *planes_, const uint16_t *coeffs_,
                                                       const uint16_t *x_, int I_, int n_tiles_, int n_gblocks_,
                                                       uint16_t *y_, int O_, GemvArgs a_rest)
{
    GemvArgs a = a_rest;
    a.planes = planes_;
    a.coeffs = coeffs_;
    a.x = x_;
    a.I = I_;
    a.n_tiles = n_tiles_;
    a.n_gblocks = n_gblocks_;
    a.y = y_;
    a.O = O_;
    gemv_b1_body<K, T, A8, IX>(a, blockIdx.x);
}

// Grouped launch (per-group coefficients; A8: SBVR-8 activations): the
// workgroups of every member in one grid, each bound to its member's matrix.
template <int K, int T, bool A8>
__global__ void __launch_bounds__(1024) gemv_b1_group_kernel(GemvArgs a_rest, GemvGroup g)
{
    GemvArgs a = a_rest;
    const unsigned bid = (unsigned)bind_group_member(g, a, (int)blockIdx.x);
    gemv_b1_body<K, T, A8, false>(a, bid);
}

// Launch shape.  T tiles (T * TR rows) per workgroup: the most (<= 8) that still
// leaves >= 256 workgroups for 256 CUs and >= 2048 wavefronts in all; one
// wavefront per gblock.  (Measured T = 1 / 2 / 4 / 8: 4096 x 4096 4.30 / 4.01 /
// 3.99 / 4.53 us, 1024 x 4096 2.76 / 2.80 / 3.24 / 4.23, 2048 x 4096 3.27 /
// 3.09 / 3.40 / 4.28, 8192 x 1024 3.59 / 3.26 / 3.45 / 3.45: the wavefront
// count picks the fastest in each.)
constexpr int B1_MAX_WAVES = 16;

static int choose_b1_tiles(const Dims &d)
{
#ifdef SBVR_TUNE_T
    return SBVR_TUNE_T;
#else
    for (int t = 8; t > 1; t >>= 1)
        if (d.n_tiles / t >= 256 && (long)(d.n_tiles / t) * d.n_gblocks >= 2048)
            return t;
    return 1;
#endif
}

template <int K, bool A8, bool IX>
static const void *b1_kernel_for(int T)
{
    switch (T) {
    case 8: return (const void *)gemv_b1_kernel<K, 8, A8, IX>;
    case 4: return (const void *)gemv_b1_kernel<K, 4, A8, IX>;
    case 2: return (const void *)gemv_b1_kernel<K, 2, A8, IX>;
    default: return (const void *)gemv_b1_kernel<K, 1, A8, IX>;
    }
}

template <int K>
static const void *b1_kernel_for(int T, bool a8, bool ix)
{
    if (ix)
        return a8 ? b1_kernel_for<K, true, true>(T) : b1_kernel_for<K, false, true>(T);
    return a8 ? b1_kernel_for<K, true, false>(T) : b1_kernel_for<K, false, false>(T);
}

// Matrices with more (tile, gblock) blocks than this, or more than 16
// gblocks per row, stream through the pipelined kernel.
#ifndef SBVR_B1S_MIN_BLOCKS
#define SBVR_B1S_MIN_BLOCKS 24576
#endif

int launch_gemv_b1(const Dims &d, const WeightRef &w, const uint16_t *x, uint16_t *y, bool a8,
                   hipStream_t stream)
{
    if (d.n_gblocks > B1_MAX_WAVES || (long)d.n_tiles * d.n_gblocks >= SBVR_B1S_MIN_BLOCKS)
        return launch_gemv_b1s(d, w, x, y, a8, stream);
    const int T = choose_b1_tiles(d);
    const int waves = d.n_gblocks;
    GemvArgs a = {(const uint4 *)w.planes, (const uint16_t *)w.coeffs, x, y, d.O, d.I, d.k,
                  d.n_tiles, d.n_gblocks, 1, 1, 0, (const uint16_t *)w.index, (const uint16_t *)w.table,
                  w.n_sets};
    const bool ix = w.index != nullptr;
    const int grid = (d.n_tiles + T - 1) / T;
    const size_t lds = (size_t)waves * B1_WAVE_LDS + (size_t)waves * T * d.tr * 4;
    const void *fn = d.k == 4   ? b1_kernel_for<4>(T, a8, ix)
                     : d.k == 3 ? b1_kernel_for<3>(T, a8, ix)
                     : d.k == 2 ? b1_kernel_for<2>(T, a8, ix)
                                : b1_kernel_for<1>(T, a8, ix);
    void *args[] = {&a.planes, &a.coeffs, &a.x, &a.I, &a.n_tiles, &a.n_gblocks, &a.y, &a.O, &a};
    return launch_kernel(fn, dim3(grid), dim3(64 * waves), lds, stream, args);
}

// the C ABI's bound, and the three comparisons of bind_group_member
static_assert(GROUP_MAX == SBVR_GEMV_GROUP_MAX && GROUP_MAX == 4, "group table size");

int fill_group(GemvGroup &g, int n, const GemvMember *mem, const Dims &d, int tiles_per_group)
{
    int wg = 0;
    for (int i = 0; i < GROUP_MAX; ++i) {
        const GemvMember &m = mem[i < n ? i : 0];
        g.planes[i] = (const uint4 *)m.planes;
        g.coeffs[i] = (const uint16_t *)m.coeffs;
        g.x[i] = m.x;
        g.y[i] = m.y;
        g.O[i] = m.O;
        g.n_tiles[i] = make_dims(m.O, d.I, d.k).n_tiles;
        g.wg0[i] = i < n ? wg : INT_MAX;
        if (i < n)
            wg += (g.n_tiles[i] + tiles_per_group - 1) / tiles_per_group;
    }
    return wg;
}

template <int K, bool A8>
static const void *b1_group_kernel_for(int T)
{
    switch (T) {
    case 8: return (const void *)gemv_b1_group_kernel<K, 8, A8>;
    case 4: return (const void *)gemv_b1_group_kernel<K, 4, A8>;
    case 2: return (const void *)gemv_b1_group_kernel<K, 2, A8>;
    default: return (const void *)gemv_b1_group_kernel<K, 1, A8>;
    }
}

template <int K>
static const void *b1_group_kernel_for(int T, bool a8)
{
    return a8 ? b1_group_kernel_for<K, true>(T) : b1_group_kernel_for<K, false>(T);
}

int launch_gemv_group(int n, const GemvMember *mem, int I, int k, bool a8, hipStream_t stream)
{
    // the combined shape (every member's row tiles) selects kernel and shape
    Dims d = make_dims(mem[0].O, I, k);
    int tiles = 0;
    for (int i = 0; i < n; ++i)
        tiles += make_dims(mem[i].O, I, k).n_tiles;
    d.n_tiles = tiles;
    d.O = tiles * d.tr;
    if (d.n_gblocks > B1_MAX_WAVES || (long)d.n_tiles * d.n_gblocks >= SBVR_B1S_MIN_BLOCKS)
        return launch_gemv_b1s_group(d, n, mem, a8, stream);
    const int T = choose_b1_tiles(d);
    const int waves = d.n_gblocks;
    GemvGroup g;
    const int grid = fill_group(g, n, mem, d, T);
    GemvArgs a = {nullptr, nullptr, nullptr, nullptr, 0, d.I, d.k, 0, d.n_gblocks, 1, 1, 0, nullptr, nullptr, 0};
    const size_t lds = (size_t)waves * B1_WAVE_LDS + (size_t)waves * T * d.tr * 4;
    const void *fn = d.k == 4   ? b1_group_kernel_for<4>(T, a8)
                     : d.k == 3 ? b1_group_kernel_for<3>(T, a8)
                     : d.k == 2 ? b1_group_kernel_for<2>(T, a8)
                                : b1_group_kernel_for<1>(T, a8);
    void *args[] = {&a, &g};
    return launch_kernel(fn, dim3(grid), dim3(64 * waves), lds, stream, args);
}

}  // namespace sbvr
