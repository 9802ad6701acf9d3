// Small-batch SBVR GEMM (B <= 8 activation vectors, Sec. 4.4 per vector):
// the weights are streamed once for all B vectors.
//
// Dense activation operands: one 16x16x128 instruction covers one group (its
// four 32-slot k-blocks are the group's four plane words) and its 16 output
// columns are (vector, limb) pairs, five vectors per column set (15 columns);
// B > 5 uses a second set.  Each lane applies the coefficients of its tile
// row to its four D rows (planes) after every instruction.
//
// Split-K inside the workgroup as in the batch-1 kernel: wavefront w owns
// gblocks [w*gpw, (w+1)*gpw); partial sums are reduced through LDS in a fixed
// order.  LDS per wavefront: limbs [group slot][vector][limb][128 bytes in
// element order] + 16 zero bytes, then the reduction buffer.
#include "device_ops.h"
#include "launch.h"

namespace sbvr {

constexpr int SB_VEC_PER_SET = 5;

__host__ __device__ constexpr int sb_wave_lds(int B) { return GB * B * 3 * GROUP + 16; }

template <int K, int T, int NS>
__global__ void __launch_bounds__(512) gemm_sb_kernel(GemvArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int B = a.B;
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int nw = blockDim.x >> 6;
    const int wave_lds = sb_wave_lds(B);
    unsigned char *lds = smem + wv * wave_lds;
    float *red = (float *)(smem + nw * wave_lds);  // [nw][T][NS][4 rows][16 cols]

    constexpr int k = K;
    const int tile0 = blockIdx.x * T;
    const int gb_begin = wv * a.gpw;
    const int gb_end = min(a.n_gblocks, gb_begin + a.gpw);
    const int zero_off = GB * B * 3 * GROUP;
    if (lane == 0)
        *(uint4 *)(lds + zero_off) = make_uint4(0u, 0u, 0u, 0u);

    // per-vector scales
    int sig[8];
    float lsc[8];
    for (int b = 0; b < 8; ++b) {
        sig[b] = 0;
        lsc[b] = 1.f;
    }
    for (int b = 0; b < B; ++b) {
        float amax = 0.f;
        for (int gb = gb_begin; gb < gb_end; ++gb) {
            const int e = gb * (GB * GROUP) + lane * 8;
            if (e < a.I)
                amax = fmaxf(amax, absmax8(*(const uint4 *)(a.x + (size_t)b * a.I + e)));
        }
        sig[b] = scale_exponent(wave_max(amax));
        lsc[b] = ldexpf(1.0f, sig[b] + inv_alpha_exp(lane & 3));
    }

    // lane roles
    const int n = lane & 15, kb = lane >> 4;
    const int col_vec = n / 3, col_limb = n % 3;
    int lo_off[NS], hi_off[NS];
#pragma unroll
    for (int st = 0; st < NS; ++st) {
        const int vec = st * SB_VEC_PER_SET + col_vec;
        const bool ok = (n < 15) && vec < B;
        const int base = (vec * 3 + col_limb) * GROUP + 16 * kb;  // + slot * B*3*128
        lo_off[st] = ok ? base : -1;
        hi_off[st] = ok ? base + 64 : -1;
    }
    const int slot_stride = B * 3 * GROUP;
    const int a_r = (lane & 15) >> 2, a_i = lane & 3, a_w = lane >> 4;
    const bool a_ok = a_i < k;
    const size_t pblk_words = plane_block_words(k);
    const size_t cblk = coeff_block_entries(k);
    const int c_row = (lane >> 4) * GB * k;  // D rows: tile row lane/16, planes 0..3
    const int wr_base = (lane >> 4) * slot_stride + 8 * (lane & 15);  // + (vec*3+limb)*128

    float acc[T][NS];
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
        for (int st = 0; st < NS; ++st)
            acc[t][st] = 0.f;

    const uint32_t *pw = (const uint32_t *)a.planes;
    for (int gb = gb_begin; gb < gb_end; ++gb) {
        // limbs of every vector for this gblock
        const int e = gb * (GB * GROUP) + lane * 8;
        for (int b = 0; b < B; ++b) {
            const uint4 xv = (e < a.I) ? *(const uint4 *)(a.x + (size_t)b * a.I + e)
                                       : make_uint4(0u, 0u, 0u, 0u);
            const Limbs L = make_limbs(xv, lsc[b]);
            unsigned char *dst = lds + wr_base + b * 3 * GROUP;
            *(uint2 *)(dst + 0 * GROUP) = make_uint2(L.hi[0], L.hi[1]);
            *(uint2 *)(dst + 1 * GROUP) = make_uint2(L.mid[0], L.mid[1]);
            *(uint2 *)(dst + 2 * GROUP) = make_uint2(L.lo[0], L.lo[1]);
        }
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const int tile = tile0 + t;
            if (tile >= a.n_tiles)
                continue;
            const size_t blk = (size_t)tile * a.n_gblocks + gb;
            const uint16_t *cb = a.coeffs + blk * cblk + c_row;
#pragma unroll
            for (int gs = 0; gs < GB; ++gs) {
                const uint32_t word =
                    a_ok ? pw[blk * pblk_words + ((gs * TILE_ROWS + a_r) * k + a_i) * 4 + a_w] : 0u;
                const v8i A = fp4_operand(word);
                const uint2 c = load_coeffs<K>(cb + gs * k);
#pragma unroll
                for (int st = 0; st < NS; ++st) {
                    const unsigned char *lo = lds + (lo_off[st] < 0 ? zero_off : lo_off[st] + gs * slot_stride);
                    const unsigned char *hi = lds + (hi_off[st] < 0 ? zero_off : hi_off[st] + gs * slot_stride);
                    const v8i Bop = lds_operand(lo, hi);
                    v4f d = {0.f, 0.f, 0.f, 0.f};
                    d = mfma_fp4_fp8(A, Bop, d);
                    acc[t][st] += apply_coeffs(c, d);
                }
            }
        }
    }

    // lane (column n, row lane/16): column n = (vector st*5 + n/3, limb n%3)
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
        for (int st = 0; st < NS; ++st) {
            const int vec = st * SB_VEC_PER_SET + col_vec;
            float v = 0.f;
            if (n < 15 && vec < B)
                v = acc[t][st] * ldexpf(1.0f, -sig[vec]);
            red[(((wv * T + t) * NS + st) * TILE_ROWS + (lane >> 4)) * 16 + n] = v;
        }
    __syncthreads();
    for (int idx = threadIdx.x; idx < T * TILE_ROWS * B; idx += blockDim.x) {
        const int vec = idx % B, tr = idx / B;
        const int t = tr / TILE_ROWS, r = tr % TILE_ROWS;
        const int o = (tile0 + t) * TILE_ROWS + r;
        if (o >= a.O)
            continue;
        const int st = vec / SB_VEC_PER_SET, cv = vec % SB_VEC_PER_SET;
        float v = 0.f;
        for (int w = 0; w < nw; ++w) {
            const float *rr = red + (((w * T + t) * NS + st) * TILE_ROWS + r) * 16 + cv * 3;
            v += rr[0];
            v += rr[1];
            v += rr[2];
        }
        a.y[(size_t)vec * a.O + o] = __half_as_ushort(__float2half_rn(v));
    }
}


// Small batch: the per-wavefront limb buffer grows with B, so the number of
// wavefronts per workgroup is capped to keep dynamic LDS within 64 KiB.
static size_t sb_red_bytes_per_wave(int T, int ns) { return (size_t)T * ns * TILE_ROWS * 16 * 4; }

struct SBConfig {
    int T, gpw, waves;
};

static SBConfig choose_sb(const Dims &d, int B)
{
    SBConfig c;
    c.T = (d.n_tiles >= 2 * 256) ? 2 : 1;
    const int ns = (B + SB_VEC_PER_SET - 1) / SB_VEC_PER_SET;
    const size_t per_wave = sb_wave_lds(B) + sb_red_bytes_per_wave(c.T, ns);
    int max_waves = (int)((64 * 1024) / per_wave);
    if (max_waves > 8)
        max_waves = 8;
    int gpw = d.n_gblocks <= 8 ? 1 : (d.n_gblocks <= 32 ? 2 : 4);
    const int min_gpw = (d.n_gblocks + max_waves - 1) / max_waves;
    if (gpw < min_gpw)
        gpw = min_gpw;
    c.gpw = gpw;
    c.waves = (d.n_gblocks + gpw - 1) / gpw;
    return c;
}

template <int K>
static const void *sb_kernel_for(int T, int ns)
{
    if (T == 2)
        return ns == 1 ? (const void *)gemm_sb_kernel<K, 2, 1> : (const void *)gemm_sb_kernel<K, 2, 2>;
    return ns == 1 ? (const void *)gemm_sb_kernel<K, 1, 1> : (const void *)gemm_sb_kernel<K, 1, 2>;
}

int launch_gemm_sb(const Dims &d, const void *planes_dev, const void *coeffs_dev,
                   const uint16_t *X, uint16_t *Y, int B, hipStream_t stream)
{
    const SBConfig c = choose_sb(d, B);
    GemvArgs a = {(const uint4 *)planes_dev, (const uint16_t *)coeffs_dev, X, Y, d.O, d.I, d.k,
                  d.n_tiles, d.n_gblocks, c.gpw, B};
    const int ns = (B + SB_VEC_PER_SET - 1) / SB_VEC_PER_SET;
    const int grid = (d.n_tiles + c.T - 1) / c.T;
    const size_t lds = (size_t)c.waves * (sb_wave_lds(B) + sb_red_bytes_per_wave(c.T, ns));
    const void *fn = d.k == 4   ? sb_kernel_for<4>(c.T, ns)
                     : d.k == 3 ? sb_kernel_for<3>(c.T, ns)
                     : d.k == 2 ? sb_kernel_for<2>(c.T, ns)
                                : sb_kernel_for<1>(c.T, ns);
    void *args[] = {&a};
    return launch_kernel(fn, dim3(grid), dim3(64 * c.waves), lds, stream, args);
}

}  // namespace sbvr
