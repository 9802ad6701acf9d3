// Streaming batch-1 SBVR GEMV (Sec. 4.4) for matrices too large to hold in
// flight at once.
//
// A workgroup owns tpw consecutive tiles (TR rows each) and every gblock
// (512 inner elements) of them; its W wavefronts split the gblocks, wavefront
// w taking w, w+W, w+2W, ...  A wavefront's work is the sequence of items
// (gblock, tile): for each of its gblocks, the workgroup's tiles in order.
// The activation operand of a gblock is built once (same block-diagonal fp8
// operand and fp4 plane operand as the one-shot kernel), then the items stream
// through a D-deep ring of registers: the loads of item m+D are issued right
// after item m is consumed, crossing into the next gblock without a pause.
//
// The ring is loaded through buffer descriptors bounded by the workgroup's
// tile range, so the loads a wavefront issues past its last item read zero and
// touch no memory: every ring slot is reloaded unconditionally and the
// compiler keeps each slot in fixed registers with counted waits.
//
// Row sums of each (tile, gblock) item are added into an LDS array
// [tile][wavefront][TR rows] in gblock order; at the end the workgroup sums the
// wavefronts in order, so the result is deterministic and no global
// workspace is used.
//
// Memory behaviour: with D = 2 a wavefront keeps up to two items (about
// 2.3 KB of weights) in flight, and 16 wavefronts per CU (512 workgroups of
// 8) keep ~36 KB per CU outstanding, while each workgroup's requests stay in
// a narrow, advancing address window.  More workgroups measured slower:
// every extra workgroup repeats the activation load and operand build, and
// shortens the stream of items that amortises them.  For the same reason
// k = 4 with at most 8 wavefronts runs one workgroup per CU with D = 4
// (about the same bytes in flight, half the builds per CU); elsewhere deeper
// rings measured slower.
#include "device_ops.h"
#include "launch.h"

namespace sbvr {

// per wavefront: [q][s][l][32 B] limb chunks, then 256 zero bytes (the
// operand halves a lane does not cover read 16 of them, a different 16 for
// each lane of a 16-lane group: reading one shared chunk from most lanes
// serialised the LDS reads, about 0.3 us on the latency-bound launches)
constexpr int B1S_WAVE_LDS = 2048 + 256;
// Ring depth: one gblock per wavefront keeps 64 VGPRs (8 wavefronts per
// SIMD) at depth 2; with several gblocks the workgroups are fewer and a
// deeper ring keeps enough bytes in flight.
#ifndef SBVR_B1S_DEPTH
#define SBVR_B1S_DEPTH 2
#endif
// With several gblocks per wavefront, a workgroup with fewer than this many
// tiles runs the depth-2 ring (a wavefront's item runs are short there and
// the shallower ring starts sooner; 8B down: 8.7 -> 8.3 us).
#ifndef SBVR_B1S_SHORT_TPW
#define SBVR_B1S_SHORT_TPW 8
#endif
#ifndef SBVR_B1S_DEPTH_MULTI
#define SBVR_B1S_DEPTH_MULTI 3
#endif
#ifndef SBVR_B1S_MAX_WAVES
#define SBVR_B1S_MAX_WAVES 16
#endif
// Workgroups per launch: with one gblock per wavefront, two resident per CU
// (half as many for workgroups of more than 8 wavefronts); one per CU
// (longer item streams per wavefront) with several gblocks per wavefront.
#ifndef SBVR_B1S_GROUPS
#define SBVR_B1S_GROUPS 512
#endif
#ifndef SBVR_B1S_GROUPS_MULTI
#define SBVR_B1S_GROUPS_MULTI 256
#endif
// k = 4 with one gblock per wavefront and at most 8 wavefronts (Llama-3-8B
// gate/up), per-group coefficients: one workgroup per CU with a depth-4 ring
// -- about the same bytes in flight as two workgroups at depth 2, and half
// the activation builds per CU (gate 7.55 -> 7.35 us, W4A8 7.87 -> 7.52; at
// k = 3 the same shape was slower, 7.73 -> 8.17).
#ifndef SBVR_B1S_GROUPS_WIDE
#define SBVR_B1S_GROUPS_WIDE 256
#endif
#ifndef SBVR_B1S_DEPTH_WIDE
#define SBVR_B1S_DEPTH_WIDE 4
#endif

// A8: activations converted online to SBVR-8.  IX: coefficient-cache format;
// each item's coefficient sets are then gathered through its index block, and
// the ring runs in three stages: the index block of item m+2D is loaded when
// item m is consumed, and the sets of item m+D are gathered then from the
// index block loaded D items earlier, so neither the index load nor the gather
// waits on anything issued less than D items before.
// The fields every wavefront needs (its first loads' addresses and sizes, the
// output and the wavefront count) come again as leading scalar arguments: the
// compiler preloads those into SGPRs at launch (built with
// -amdgpu-kernarg-preload-count), so neither the first loads nor the LDS
// waits before the matrix-core work sit behind a kernel-argument fetch (a
// scalar load shares the LDS wait counter); the rest are read from the struct.
// a * b rounded to binary32 on its own: never fused with a later addition
__device__ __forceinline__ float mul_rounded(float a, float b)
{
#pragma clang fp contract(off)
    return a * b;
}

// The kernel body for workgroup `bid` (of nw wavefronts) of the matrix in `a`.
template <int K, int D, bool MULTI, bool A8, bool IX>
__device__ __forceinline__ void gemv_b1s_body(const GemvArgs &a, int nw, unsigned bid)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63;
    const int wv = wave_id();
    unsigned char *lds = smem + wv * B1S_WAVE_LDS;
    constexpr int TR = tile_rows(K), NP = partials_per_lane<K>();
    float *red = (float *)(smem + nw * B1S_WAVE_LDS);  // [tpw][nw][TR]

    const int tile0 = bid * a.tpw;
    const int ntl = min(a.tpw, a.n_tiles - tile0);
    // MULTI: several gblocks per wavefront; otherwise exactly one (wv)
    const int n_items = MULTI ? ((a.n_gblocks - wv + nw - 1) / nw) * ntl : ntl;

    // A operand lane mapping: row m = lane%16 = (tile row, plane), k-block =
    // group slot; empty plane slots (K = 3) read a valid slot and are zeroed.
    bool a_ok;
    const unsigned p_lane = a_slot_bytes<K>(lane, a_ok);
    // coefficients of the lane's D rows (group slot (lane%16)/4)
    const unsigned c_lane = (unsigned)(((lane >> 4) * GB + ((lane & 15) >> 2)) * coefs_per_lane<K>()) * 2u;
    constexpr unsigned PBLK_B = GB * TR * K * 16;  // bytes per plane block
    constexpr unsigned CBLK_B = GB * TR * K * 2;   // bytes per coefficient block
    const unsigned pstep = (unsigned)a.n_gblocks * PBLK_B;  // next tile, same gblock
    const unsigned cstep = (unsigned)a.n_gblocks * CBLK_B;
    const size_t blk0 = (size_t)tile0 * a.n_gblocks;
    const buf_rsrc prs = make_rsrc((const unsigned char *)a.planes + blk0 * PBLK_B, (unsigned)ntl * pstep);
    const buf_rsrc crs = make_rsrc((const unsigned char *)a.coeffs + blk0 * CBLK_B, (unsigned)ntl * cstep);

    // coefficient-cache format: index blocks (same block order) and the table
    constexpr unsigned IBLK_B = GB * TR * 2;  // bytes per index block
    const unsigned istep = (unsigned)a.n_gblocks * IBLK_B;
    const unsigned i_lane = (unsigned)(((lane >> 4) * GB + ((lane & 15) >> 2)) * index_per_lane(K)) * 2u;
    buf_rsrc irs, trs;
    if constexpr (IX) {
        irs = make_rsrc((const unsigned char *)a.index + blk0 * IBLK_B, (unsigned)ntl * istep);
        trs = make_rsrc(a.table, (unsigned)a.n_sets * (TABLE_STRIDE * 2));
    }

    // Cursor (wavefront-uniform) over the wavefront's items: returns the item's
    // block offset in units of blocks-per-tile (tile i * n_gblocks + gblock) or
    // -1 past the end (MULTI; without MULTI, items past the last tile fall
    // outside the descriptors' range by themselves).
    auto advance = [&](int &ci, int &cg, unsigned &po, unsigned &co, unsigned &io) {
        if constexpr (MULTI) {
            po = co = io = BUF_OOB;
            if (cg < a.n_gblocks) {
                po = (unsigned)ci * pstep + (unsigned)cg * PBLK_B;
                co = (unsigned)ci * cstep + (unsigned)cg * CBLK_B;
                io = (unsigned)ci * istep + (unsigned)cg * IBLK_B;
            }
            if (++ci == ntl) {
                ci = 0;
                cg += nw;
            }
        } else {
            po = (unsigned)ci * pstep + (unsigned)wv * PBLK_B;
            co = (unsigned)ci * cstep + (unsigned)wv * CBLK_B;
            io = (unsigned)ci * istep + (unsigned)wv * IBLK_B;
            ++ci;
        }
    };
    // Prefetch cursors: next item whose planes (and coefficients) are loaded,
    // and, for IX, next item whose index block is loaded (D items further).
    int pf_i = 0, pf_gb = wv, ix_i = 0, ix_gb = wv;
    uint4 P[D];
    uint2 C[D];
    typename IxLane<K>::type IXr[D];
    auto load_ix = [&](int j) {
        unsigned po, co, io;
        advance(ix_i, ix_gb, po, co, io);
        IXr[j] = buf_index<K>(irs, i_lane + io);
    };
    auto gather = [&](int j) { C[j] = table_coefs4<K>(trs, IXr[j]); };
    auto issue = [&](int j) {
        unsigned po, co, io;
        advance(pf_i, pf_gb, po, co, io);
        P[j] = buf_load16(prs, p_lane + po);
        if constexpr (IX) {
            __builtin_amdgcn_sched_barrier(0);
            gather(j);  // the sets of this item (index loaded D items ago)
            __builtin_amdgcn_sched_barrier(0);
            load_ix(j);                           // index block D items further on
        } else {
            C[j] = buf_coefs4<K>(crs, c_lane + co);
        }
    };
    // Activations of a gblock; lanes past I (ragged end) read a valid address
    // and are zeroed when the operand is built.
    auto load_x = [&](int gb) {
        const int e = gb * (GB * GROUP) + lane * 8;
        return *(const uint4 *)(a.x + min(e, a.I - 8));
    };

    // x first: the operand build waits only for it, not for the ring loads
    uint4 x_cur = load_x(wv);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (IX) {
        // first D index blocks, then the first D items' planes; only then the
        // gathers that wait for those index blocks (and the next D index blocks)
#pragma unroll
        for (int j = 0; j < D; ++j)
            load_ix(j);
#pragma unroll
        for (int j = 0; j < D; ++j) {
            unsigned po, co, io;
            advance(pf_i, pf_gb, po, co, io);
            P[j] = buf_load16(prs, p_lane + po);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < D; ++j) {
            gather(j);
            __builtin_amdgcn_sched_barrier(0);
            load_ix(j);
            __builtin_amdgcn_sched_barrier(0);
        }
    } else {
        // in the loop's order (planes, coefficients per item): the compiler's
        // counted waits at the loop head then match on both incoming paths
#pragma unroll
        for (int j = 0; j < D; ++j) {
            issue(j);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    uint4 x_next;
    if constexpr (MULTI)
        x_next = load_x(wv + nw);
    __builtin_amdgcn_sched_barrier(0);

    // B operand lane mapping (see the one-shot kernel): column n = lane%16 =
    // (slot s, limb l), k-block lane/16.
    const int wr_off = ((((lane & 15) >> 2) * 4 + (lane >> 4)) * 4) * 32 + 8 * (lane & 3);
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
    *(uint32_t *)(lds + 2048 + 4 * lane) = 0u;  // the zero region

    v8i Bq[4];
    float inv_scale;
    auto build = [&](uint4 xr, int gb) {
        const uint4 xv = gb * (GB * GROUP) + lane * 8 < a.I ? xr : make_uint4(0u, 0u, 0u, 0u);
        Limbs L;
        if constexpr (A8) {
            L = a8_limbs(xv, lane, inv_alpha, inv_scale);  // per lane: its column's group scale
        } else {
            const int sigma = scale_exponent(wave_absmax_h(xv));
            inv_scale = ldexpf(1.0f, -sigma);
            L = split_limbs(xv, sigma, inv_alpha);
        }
        // same wavefront: these writes land before the reads below, and after
        // the reads of the previous gblock's operand
#pragma unroll
        for (int j = 0; j < (A8 ? 2 : 4); ++j)
            *(uint2 *)(lds + wr_off + j * 32) = make_uint2(L.l[j][0], L.l[j][1]);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            Bq[q] = lds_operand(lds + lo_off + q * lo_step, lds + hi_off + q * hi_step);
    };
    build(x_cur, wv);
    __builtin_amdgcn_sched_barrier(0);

    float *red_w = red + wv * TR + (lane >> 4) * NP;
    int cur_i = 0, cur_gb = wv;
    for (int m0 = 0; m0 < n_items; m0 += D) {
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int m = m0 + j;
            if (m < n_items) {
                if constexpr (MULTI) {
                    if (cur_i == 0 && m > 0) {  // first item of the next gblock
                        build(x_next, cur_gb);
                        x_next = load_x(cur_gb + nw);
                    }
                }
                const uint4 pw = a_ok ? P[j] : make_uint4(0u, 0u, 0u, 0u);
                v4f d = {0.f, 0.f, 0.f, 0.f};
                d = mfma_fp4_fp8<A8>(fp4_operand(pw.x), Bq[0], d);
                d = mfma_fp4_fp8<A8>(fp4_operand(pw.y), Bq[1], d);
                d = mfma_fp4_fp8<A8>(fp4_operand(pw.z), Bq[2], d);
                d = mfma_fp4_fp8<A8>(fp4_operand(pw.w), Bq[3], d);
                float part[NP];
                apply_coefs<K>(C[j], d, part);
                // the scaled partial is rounded before the row sum (no fused
                // multiply-add with a neighbour's term), as in the one-shot
                // kernel: with SBVR-8 activations the scale is not a power of
                // two, and both kernels then give the same bits
#pragma unroll
                for (int p = 0; p < NP; ++p)
                    part[p] = row16_sum(mul_rounded(part[p], inv_scale));
                if ((lane & 15) == 0) {
                    float *r = red_w + cur_i * nw * TR;
#pragma unroll
                    for (int p = 0; p < NP; ++p) {
                        if (!MULTI || cur_gb == wv)
                            r[p] = part[p];
                        else
                            r[p] += part[p];
                    }
                }
                if (++cur_i == ntl && MULTI) {
                    cur_i = 0;
                    cur_gb += nw;
                }
            }
            issue(j);
        }
    }

    __syncthreads();
    const int row_base = tile0 * TR;
    for (int idx = threadIdx.x; idx < ntl * TR; idx += 64 * nw) {
        const int o = row_base + idx;
        if (o < a.O) {
            const float *r = red + (idx / TR) * nw * TR + (idx % TR);
            float v = 0.f;
            for (int w = 0; w < nw; ++w)
                v += r[w * TR];
            a.y[o] = __half_as_ushort(__float2half_rn(v));
        }
    }
}

template <int K, int D, bool MULTI, bool A8, bool IX>
__global__ void __launch_bounds__(1024) gemv_b1s_kernel(const uint4 *planes_, const uint16_t *coeffs_,
                                                        const uint16_t *x_, int I_, int n_tiles_, int n_gblocks_, int tpw_,
                                                        uint16_t *y_, int O_, int nw_, GemvArgs a_rest)
{
    GemvArgs a = a_rest;
    a.planes = planes_;
    a.coeffs = coeffs_;
    a.x = x_;
    a.I = I_;
    a.n_tiles = n_tiles_;
    a.n_gblocks = n_gblocks_;
    a.tpw = tpw_;
    a.y = y_;
    a.O = O_;
    gemv_b1s_body<K, D, MULTI, A8, IX>(a, nw_, blockIdx.x);
}

// Grouped launch (per-group coefficients; A8: SBVR-8 activations): the
// workgroups of every member in one grid, each bound to its member's matrix.
template <int K, int D, bool MULTI, bool A8>
__global__ void __launch_bounds__(1024) gemv_b1s_group_kernel(int nw_, GemvArgs a_rest, GemvGroup g)
{
    GemvArgs a = a_rest;
    const unsigned bid = (unsigned)bind_group_member(g, a, (int)blockIdx.x);
    gemv_b1s_body<K, D, MULTI, A8, false>(a, nw_, bid);
}

template <int K, bool A8, bool IX>
static const void *b1s_kernel_for(bool multi, bool short_run, bool wide)
{
    if constexpr (K == 4 && !IX) {
        if (wide)
            return (const void *)gemv_b1s_kernel<K, SBVR_B1S_DEPTH_WIDE, false, A8, IX>;
    }
    if (!multi)
        return (const void *)gemv_b1s_kernel<K, SBVR_B1S_DEPTH, false, A8, IX>;
    return short_run ? (const void *)gemv_b1s_kernel<K, 2, true, A8, IX>
                     : (const void *)gemv_b1s_kernel<K, SBVR_B1S_DEPTH_MULTI, true, A8, IX>;
}

template <int K>
static const void *b1s_kernel_for(bool multi, bool short_run, bool wide, bool a8, bool ix)
{
    if (ix)
        return a8 ? b1s_kernel_for<K, true, true>(multi, short_run, wide)
                  : b1s_kernel_for<K, false, true>(multi, short_run, wide);
    return a8 ? b1s_kernel_for<K, true, false>(multi, short_run, wide)
              : b1s_kernel_for<K, false, false>(multi, short_run, wide);
}

// Launch shape of the streaming kernel for the (combined) shape d.
struct B1sShape {
    int waves, tpw, gpw;
    bool multi, short_run, wide;
    size_t lds;
};

static B1sShape b1s_shape(const Dims &d, bool ix)
{
    B1sShape sh;
    sh.gpw = (d.n_gblocks + SBVR_B1S_MAX_WAVES - 1) / SBVR_B1S_MAX_WAVES;
    // with several gblocks per wavefront, always the full 16 wavefronts: the
    // strided gblock assignment then gives every SIMD (wavefronts w, w + 4, ..)
    // the same number of gblocks to within one (8B down, 28 gblocks: 14
    // wavefronts left two SIMDs with 8 gblocks and two with 6; 9.1 -> 8.2 us;
    // 70B down 24.7 -> 22.3 us)
    sh.waves = sh.gpw > 1 ? SBVR_B1S_MAX_WAVES : (d.n_gblocks + sh.gpw - 1) / sh.gpw;
    // one gblock per wavefront: about 16 wavefronts per CU -- 512 workgroups of
    // up to 8 wavefronts, 256 of more (70B q/o, gate/up: 8.4 -> 8.1 us,
    // 22.3 -> 22.1 us) -- except the k = 4 depth-4 launch (256 of up to 8)
    sh.wide = d.k == 4 && sh.gpw == 1 && sh.waves <= 8 && !ix;
    const int groups = sh.gpw > 1 ? SBVR_B1S_GROUPS_MULTI
                       : sh.wide  ? SBVR_B1S_GROUPS_WIDE
                                  : (sh.waves > 8 ? SBVR_B1S_GROUPS / 2 : SBVR_B1S_GROUPS);
    // tiles per workgroup, capped so that the dynamic LDS (operand staging
    // plus the [tile][wavefront][row] sums) stays within SBVR_MAX_DYN_LDS:
    // very tall matrices get more workgroups instead
    const size_t per_tile = (size_t)sh.waves * d.tr * 4;
    const int max_tpw = (int)((SBVR_MAX_DYN_LDS - (size_t)sh.waves * B1S_WAVE_LDS) / per_tile);
    sh.tpw = min((d.n_tiles + groups - 1) / groups, max_tpw);
    sh.lds = (size_t)sh.waves * B1S_WAVE_LDS + (size_t)sh.tpw * per_tile;
    sh.multi = sh.gpw > 1;
    sh.short_run = sh.tpw < SBVR_B1S_SHORT_TPW;
    return sh;
}

int launch_gemv_b1s(const Dims &d, const WeightRef &w, const uint16_t *x, uint16_t *y, bool a8,
                    hipStream_t stream)
{
    const bool ix = w.index != nullptr;
    const B1sShape sh = b1s_shape(d, ix);
    const int grid = (d.n_tiles + sh.tpw - 1) / sh.tpw;
    GemvArgs a = {(const uint4 *)w.planes, (const uint16_t *)w.coeffs, x, y, d.O, d.I, d.k,
                  d.n_tiles, d.n_gblocks, sh.gpw, 1, sh.tpw, (const uint16_t *)w.index, (const uint16_t *)w.table,
                  w.n_sets};
    const void *fn = d.k == 4   ? b1s_kernel_for<4>(sh.multi, sh.short_run, sh.wide, a8, ix)
                     : d.k == 3 ? b1s_kernel_for<3>(sh.multi, sh.short_run, sh.wide, a8, ix)
                     : d.k == 2 ? b1s_kernel_for<2>(sh.multi, sh.short_run, sh.wide, a8, ix)
                                : b1s_kernel_for<1>(sh.multi, sh.short_run, sh.wide, a8, ix);
    int nw = sh.waves;
    void *args[] = {&a.planes, &a.coeffs, &a.x, &a.I, &a.n_tiles, &a.n_gblocks, &a.tpw, &a.y, &a.O, &nw, &a};
    return launch_kernel(fn, dim3(grid), dim3(64 * sh.waves), sh.lds, stream, args);
}

// the same instance choice as b1s_kernel_for, for the grouped kernel
template <int K, bool A8>
static const void *b1s_group_kernel_for(bool multi, bool short_run, bool wide)
{
    if constexpr (K == 4) {
        if (wide)
            return (const void *)gemv_b1s_group_kernel<K, SBVR_B1S_DEPTH_WIDE, false, A8>;
    }
    if (!multi)
        return (const void *)gemv_b1s_group_kernel<K, SBVR_B1S_DEPTH, false, A8>;
    return short_run ? (const void *)gemv_b1s_group_kernel<K, 2, true, A8>
                     : (const void *)gemv_b1s_group_kernel<K, SBVR_B1S_DEPTH_MULTI, true, A8>;
}

template <int K>
static const void *b1s_group_kernel_for(bool multi, bool short_run, bool wide, bool a8)
{
    return a8 ? b1s_group_kernel_for<K, true>(multi, short_run, wide)
              : b1s_group_kernel_for<K, false>(multi, short_run, wide);
}

int launch_gemv_b1s_group(const Dims &d, int n, const GemvMember *mem, bool a8, hipStream_t stream)
{
    const B1sShape sh = b1s_shape(d, false);
    GemvGroup g;
    const int grid = fill_group(g, n, mem, d, sh.tpw);
    GemvArgs a = {nullptr, nullptr, nullptr, nullptr, 0, d.I, d.k, 0, d.n_gblocks, sh.gpw, 1, sh.tpw,
                  nullptr, nullptr, 0};
    const void *fn = d.k == 4   ? b1s_group_kernel_for<4>(sh.multi, sh.short_run, sh.wide, a8)
                     : d.k == 3 ? b1s_group_kernel_for<3>(sh.multi, sh.short_run, sh.wide, a8)
                     : d.k == 2 ? b1s_group_kernel_for<2>(sh.multi, sh.short_run, sh.wide, a8)
                                : b1s_group_kernel_for<1>(sh.multi, sh.short_run, sh.wide, a8);
    int nw = sh.waves;
    void *args[] = {&nw, &a, &g};
    return launch_kernel(fn, dim3(grid), dim3(64 * sh.waves), sh.lds, stream, args);
}

}  // namespace sbvr
