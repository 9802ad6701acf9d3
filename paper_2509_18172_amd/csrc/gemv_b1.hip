// Batch-1 SBVR GEMV (Sec. 4.4): y[o] = sum_g sum_i c[o][g][i] * S[o][g][i].
//
// Work decomposition.  A workgroup owns T tiles (4T consecutive rows); its
// wavefront w owns gblocks [w*gpw, (w+1)*gpw) of the inner dimension (split-K
// inside the workgroup).  Partial row sums are reduced across wavefronts in
// LDS in a fixed order: results are deterministic and there is no global
// workspace.
//
// Block-diagonal activation operand.  One 16x16x128 instruction takes, in its
// four 32-slot k-blocks, word q of four different groups (the four groups of a
// gblock), and the 16 output columns are (group slot s, limb l): column 4s+l
// holds limb l of group s's activations in k-block s and zeros elsewhere.
// Four chained instructions (q = 0..3) therefore leave in D[row][4s+l] the
// complete per-plane sum of group s for limb l, and the coefficients are
// applied once per four instructions: D rows are (tile row, plane), so a lane
// multiplies its four D values by the four coefficients of one (row, group).
//
// Latency hiding.  The activations of the first gblock are loaded first and
// the T tiles' plane and coefficient blocks right after, so the wait for the
// activations leaves every weight load in flight.  Two register sets
// alternate: while one gblock is computed from set A, the next gblock's loads
// land in set B.
#include "device_ops.h"
#include "launch.h"

namespace sbvr {

constexpr int B1_WAVE_LDS = 2048;  // per wavefront: [q][s][l][32 B]

template <int K, int T>
struct B1Regs {
    uint4 p[T];  // plane words of each tile (this lane's 16 bytes)
    uint2 c[T];  // this lane's coefficients of each tile
    uint4 x;     // this lane's 8 activations
};

template <int K, int T>
__global__ void __launch_bounds__(512) gemv_b1_kernel(GemvArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63;
    const int wv = wave_id();
    const int nw = blockDim.x >> 6;
    unsigned char *lds = smem + wv * B1_WAVE_LDS;
    float *red = (float *)(smem + nw * B1_WAVE_LDS);

    const int tile0 = blockIdx.x * T;
    const int gb_begin = wv * a.gpw;
    const int gb_end = min(a.n_gblocks, gb_begin + a.gpw);

    // A operand: row m = lane%16 = (tile row r, plane i), k-block = group slot.
    // Lanes of planes >= K read a valid slot and zero it.
    const int a_r = (lane & 15) >> 2, a_i = lane & 3, a_b = lane >> 4;
    const bool a_ok = a_i < K;
    const unsigned a_off = (unsigned)((a_b * TILE_ROWS + a_r) * K + (a_ok ? a_i : 0));
    // coefficients: D rows of this lane are tile row lane/16, planes 0..3
    const unsigned c_off = (unsigned)(((lane >> 4) * GB + ((lane & 15) >> 2)) * K);
    constexpr int PBLK = GB * TILE_ROWS * K;  // uint4 per plane block
    constexpr int CBLK = TILE_ROWS * GB * K;  // coefficients per block
    // Tiles past the end (last workgroup) re-read the last tile; their rows
    // are >= O and never stored.  Block indices are wavefront-uniform, so each
    // load is a scalar base plus the lane's 32-bit offset.
    int tblk[T];
#pragma unroll
    for (int t = 0; t < T; ++t)
        tblk[t] = min(tile0 + t, a.n_tiles - 1) * a.n_gblocks;

    auto fetch = [&](int gb, B1Regs<K, T> &R) {
        // activations first; a gblock past I (ragged end) reads as zero
        const int e0 = gb * (GB * GROUP);
        if (e0 + GB * GROUP <= a.I) {
            R.x = *(const uint4 *)(a.x + e0 + lane * 8);
        } else {
            const int e = e0 + lane * 8;
            const uint4 v = *(const uint4 *)(a.x + min(e, a.I - 8));
            R.x = e < a.I ? v : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const size_t blk = (size_t)(tblk[t] + gb);
            const uint4 v = (a.planes + blk * PBLK)[a_off];
            R.p[t] = a_ok ? v : make_uint4(0u, 0u, 0u, 0u);
            R.c[t] = load_coeffs<K>(a.coeffs + blk * CBLK + c_off);
        }
    };

    // zero the limb-3 chunks: they feed the unused 4th column of each slot
    *(uint2 *)(lds + ((lane >> 2) * 4 + 3) * 32 + 8 * (lane & 3)) = make_uint2(0u, 0u);

    // limb writes: lane owns elements 8*lane .. 8*lane+7 of the gblock:
    // group slot lane/16, word (lane%16)/4, k-slots 8*(lane%4) ..
    const int wr_off = ((((lane & 15) >> 2) * 4 + (lane >> 4)) * 4) * 32 + 8 * (lane & 3);
    // B-operand reads: column n = lane%16 = (slot s, limb l), k-block lane/16.
    // fp8 k-blocks: registers 0-3 hold k = 16 kb + [0,16), registers 4-7 hold
    // k = 64 + 16 kb + [0,16); slot s covers k = 32 s + [0,32).
    const int n = lane & 15, kb = lane >> 4;
    const int s = n >> 2, l = n & 3;
    const bool act = (l < 3) && ((kb >> 1) == (s & 1));
    const int data_off = (s * 4 + l) * 32 + 16 * (kb & 1);
    const int zero_off = (s * 4 + 3) * 32;
    const int lo_off = (act && s < 2) ? data_off : zero_off;
    const int hi_off = (act && s >= 2) ? data_off : zero_off;
    const int inv_alpha = inv_alpha_exp(lane & 3);

    float acc[T];
#pragma unroll
    for (int t = 0; t < T; ++t)
        acc[t] = 0.f;

    // One gblock from register set R.
    auto compute = [&](const B1Regs<K, T> &R) {
        // per-gblock power-of-two activation scale and exact fp8 limbs
        const int sigma = scale_exponent(wave_max(absmax8(R.x)));
        const float inv_scale = ldexpf(1.0f, -sigma);
        const Limbs L = make_limbs(R.x, ldexpf(1.0f, sigma + inv_alpha));
        // same wavefront: the LDS writes complete before the reads below
        *(uint2 *)(lds + wr_off + 0 * 32) = make_uint2(L.hi[0], L.hi[1]);
        *(uint2 *)(lds + wr_off + 1 * 32) = make_uint2(L.mid[0], L.mid[1]);
        *(uint2 *)(lds + wr_off + 2 * 32) = make_uint2(L.lo[0], L.lo[1]);
        v8i Bq[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            Bq[q] = lds_operand(lds + lo_off + q * 512, lds + hi_off + q * 512);
#pragma unroll
        for (int t = 0; t < T; ++t) {
            v4f d = {0.f, 0.f, 0.f, 0.f};
            d = mfma_fp4_fp8(fp4_operand(R.p[t].x), Bq[0], d);
            d = mfma_fp4_fp8(fp4_operand(R.p[t].y), Bq[1], d);
            d = mfma_fp4_fp8(fp4_operand(R.p[t].z), Bq[2], d);
            d = mfma_fp4_fp8(fp4_operand(R.p[t].w), Bq[3], d);
            acc[t] = fmaf(apply_coeffs(R.c[t], d), inv_scale, acc[t]);
        }
    };

    if (gb_begin < gb_end) {
        B1Regs<K, T> RA, RB;
        fetch(gb_begin, RA);
        for (int gb = gb_begin;; gb += 2) {
            if (gb + 1 < gb_end)
                fetch(gb + 1, RB);
            compute(RA);
            if (gb + 1 >= gb_end)
                break;
            if (gb + 2 < gb_end)
                fetch(gb + 2, RA);
            compute(RB);
            if (gb + 2 >= gb_end)
                break;
        }
    }

    // sum the 16 columns (group slot x limb) of each row ...
#pragma unroll
    for (int t = 0; t < T; ++t)
        acc[t] = row16_sum(acc[t]);
    const int row_base = tile0 * TILE_ROWS;
    if (nw == 1) {  // inner dimension not split: store directly
        if ((lane & 15) == 0) {
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const int o = row_base + t * TILE_ROWS + (lane >> 4);
                if (o < a.O)
                    a.y[o] = __half_as_ushort(__float2half_rn(acc[t]));
            }
        }
        return;
    }
    // ... then the wavefronts, in wavefront order
    if ((lane & 15) == 0) {
#pragma unroll
        for (int t = 0; t < T; ++t)
            red[(wv * T + t) * TILE_ROWS + (lane >> 4)] = acc[t];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < T * TILE_ROWS; idx += blockDim.x) {
        const int o = row_base + idx;
        if (o < a.O) {
            float v = 0.f;
            for (int w = 0; w < nw; ++w)
                v += red[w * T * TILE_ROWS + idx];
            a.y[o] = __half_as_ushort(__float2half_rn(v));
        }
    }
}

struct B1Config {
    int T, gpw, waves;
};

// Launch shape.  T tiles (4T rows) per workgroup: the most (<= 8) that still
// leaves >= 256 workgroups for 256 CUs.  gpw gblocks per wavefront: enough
// that the grid's wavefronts fit in about one residency round, and at most 8
// wavefronts per workgroup.
#ifndef SBVR_RESIDENT_WAVES
#define SBVR_RESIDENT_WAVES 3072
#endif

static B1Config choose_b1(const Dims &d)
{
    B1Config c;
    c.T = 1;
    for (int t = 8; t > 1; t >>= 1)
        if (d.n_tiles / t >= 256) {
            c.T = t;
            break;
        }
#ifdef SBVR_TUNE_T
    c.T = SBVR_TUNE_T;
#endif
    const long grid = (d.n_tiles + c.T - 1) / c.T;
    int gpw = (int)((grid * d.n_gblocks + SBVR_RESIDENT_WAVES - 1) / SBVR_RESIDENT_WAVES);
#ifdef SBVR_TUNE_GPW
    gpw = SBVR_TUNE_GPW;
#endif
    const int min_gpw = (d.n_gblocks + 7) / 8;
    if (gpw < min_gpw)
        gpw = min_gpw;
    if (gpw < 1)
        gpw = 1;
    c.gpw = gpw;
    c.waves = (d.n_gblocks + gpw - 1) / gpw;
    return c;
}

template <int K>
static const void *b1_kernel_for(int T)
{
    switch (T) {
    case 8: return (const void *)gemv_b1_kernel<K, 8>;
    case 4: return (const void *)gemv_b1_kernel<K, 4>;
    case 2: return (const void *)gemv_b1_kernel<K, 2>;
    default: return (const void *)gemv_b1_kernel<K, 1>;
    }
}

int launch_gemv_b1(const Dims &d, const void *planes_dev, const void *coeffs_dev,
                   const uint16_t *x, uint16_t *y, hipStream_t stream)
{
    GemvArgs a = {(const uint4 *)planes_dev, (const uint16_t *)coeffs_dev, x, y, d.O, d.I, d.k,
                  d.n_tiles, d.n_gblocks, 1, 1};
    const B1Config c = choose_b1(d);
    a.gpw = c.gpw;
    const int grid = (d.n_tiles + c.T - 1) / c.T;
    const size_t lds = (size_t)c.waves * B1_WAVE_LDS + (size_t)c.waves * c.T * TILE_ROWS * 4;
    const void *fn = d.k == 4   ? b1_kernel_for<4>(c.T)
                     : d.k == 3 ? b1_kernel_for<3>(c.T)
                     : d.k == 2 ? b1_kernel_for<2>(c.T)
                                : b1_kernel_for<1>(c.T);
    void *args[] = {&a};
    return launch_kernel(fn, dim3(grid), dim3(64 * c.waves), lds, stream, args);
}

}  // namespace sbvr
