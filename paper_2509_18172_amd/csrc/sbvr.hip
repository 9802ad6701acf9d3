// SBVR GEMV for MI355X (gfx950): C ABI, repacking kernels and the matrix-core
// GEMV kernels.
//
// What is computed (Sec. 4.4): for each output row o,
//     y[o] = sum_g sum_i c[o][g][i] * S[o][g][i],   S = sum_{j in plane i} x[128 g + j]
// directly on the bit planes, without materialising decoded weights.
//
// How it maps to CDNA4.  The per-plane masked sums S are a bit-matrix times
// vector product.  Each 32-bit plane word becomes, with four mask operations,
// an fp4 (E2M1) matrix-core operand whose nibbles are 0 or a power of two
// (0.5, 1, 2, 2 for the four nibble bit positions), so the bits never have to
// be expanded element by element.  The activation side is an fp8 (E4M3)
// operand: each binary16 x is split exactly into three E4M3 limbs
// (x' = hi + mid + lo after a power-of-two scale), so the fp4 x fp8 product
// accumulated in fp32 by v_mfma_scale_f32_16x16x128_f8f6f4 reproduces the
// binary16 activations.  The matrix core therefore does the AND/popcount-like
// reduction of Sec. 4.4 on 2048 weight bits per instruction, and the vector
// ALUs only form operands and apply the coefficients (a K-times-fewer multiply
// count, as in Sec. 4.4's FMA argument).
//
// Batch 1 uses a block-diagonal activation operand: the four k-blocks of one
// instruction carry four different groups and the 16 output columns are
// (group slot, limb), so a 4 x 16 bit tile of four groups is reduced by four
// chained instructions before the coefficients are applied once.
// Small batch uses dense activation operands whose columns are
// (vector, limb) pairs, five vectors per instruction.
//
// Split-K is done inside a workgroup: each wavefront owns a contiguous range
// of 512-element blocks of the inner dimension for the workgroup's rows, and
// the partial sums are reduced through LDS in a fixed order, so results are
// deterministic and no global workspace is needed.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "layout.h"
#include "sbvr.h"

namespace sbvr {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

// --------------------------------------------------------------------------
// Repacking (canonical <-> device), one thread per 32-bit word / coefficient.
// --------------------------------------------------------------------------

__global__ void pack_planes_kernel(Dims d, const uint32_t *__restrict__ canon,
                                   uint32_t *__restrict__ dev, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const size_t bw = plane_block_words(d.k);
    const size_t blk = idx / bw;
    const int within = (int)(idx % bw);
    const int slot = within / 4, w = within % 4;
    const int i = slot % d.k, br = slot / d.k;
    const int r = br % TILE_ROWS, b = br / TILE_ROWS;
    const int o = (int)(blk / d.n_gblocks) * TILE_ROWS + r;
    const int g = (int)(blk % d.n_gblocks) * GB + b;
    uint32_t v = 0;
    if (o < d.O && g < d.G)
        v = to_device_word(canon[(((size_t)o * d.G + g) * d.k + i) * 4 + w]);
    dev[idx] = v;
}

__global__ void unpack_planes_kernel(Dims d, const uint32_t *__restrict__ dev,
                                     uint32_t *__restrict__ canon, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int w = (int)(idx % 4);
    const size_t rest = idx / 4;
    const int i = (int)(rest % d.k);
    const size_t og = rest / d.k;
    const int g = (int)(og % d.G), o = (int)(og / d.G);
    const size_t blk = (size_t)(o / TILE_ROWS) * d.n_gblocks + g / GB;
    const int slot = ((g % GB) * TILE_ROWS + o % TILE_ROWS) * d.k + i;
    canon[idx] = to_canonical_word(dev[blk * plane_block_words(d.k) + slot * 4 + w]);
}

__global__ void pack_coeffs_kernel(Dims d, const uint16_t *__restrict__ canon,
                                   uint16_t *__restrict__ dev, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const size_t be = coeff_block_entries(d.k);
    const size_t blk = idx / be;
    const int within = (int)(idx % be);
    const int i = within % d.k, rb = within / d.k;
    const int b = rb % GB, r = rb / GB;
    const int o = (int)(blk / d.n_gblocks) * TILE_ROWS + r;
    const int g = (int)(blk % d.n_gblocks) * GB + b;
    uint16_t v = 0;
    if (o < d.O && g < d.G)
        v = canon[((size_t)o * d.G + g) * d.k + i];
    dev[idx] = v;
}

__global__ void unpack_coeffs_kernel(Dims d, const uint16_t *__restrict__ dev,
                                     uint16_t *__restrict__ canon, size_t total)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int i = (int)(idx % d.k);
    const size_t og = idx / d.k;
    const int g = (int)(og % d.G), o = (int)(og / d.G);
    const size_t blk = (size_t)(o / TILE_ROWS) * d.n_gblocks + g / GB;
    canon[idx] = dev[blk * coeff_block_entries(d.k) + ((o % TILE_ROWS) * GB + g % GB) * d.k + i];
}

// --------------------------------------------------------------------------
// Operand formation.
// --------------------------------------------------------------------------

// fp4 A operand from one device plane word: register v holds, in nibble p,
// element 8v+p of the word as 0 or alpha_v, alpha = (0.5, 1, 2, 2).
__device__ __forceinline__ v8i fp4_operand(uint32_t w)
{
    v8i a;
    a[0] = (int)(w & 0x11111111u);
    a[1] = (int)(w & 0x22222222u);
    a[2] = (int)(w & 0x44444444u);
    a[3] = (int)((w >> 1) & 0x44444444u);
    a[4] = 0;
    a[5] = 0;
    a[6] = 0;
    a[7] = 0;
    return a;
}

// 1/alpha_v as a power-of-two exponent, v = (element index within word) / 8.
__device__ __forceinline__ int inv_alpha_exp(int v) { return v == 0 ? 1 : (v == 1 ? 0 : -1); }

__device__ __forceinline__ float half_bits_to_float(uint32_t bits16)
{
    return __half2float(__ushort_as_half((unsigned short)bits16));
}

__device__ __forceinline__ float absmax8(uint4 v)
{
    float m = 0.f;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        m = fmaxf(m, fabsf(half_bits_to_float(w[i] & 0xffffu)));
        m = fmaxf(m, fabsf(half_bits_to_float(w[i] >> 16)));
    }
    return m;
}

__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v = fmaxf(v, __shfl_xor(v, off));
    return v;
}

// Power-of-two exponent s with max|x| * 2^s in [64, 128): the scaled
// activations (times 1/alpha <= 2) stay below the E4M3 maximum of 448.
__device__ __forceinline__ int scale_exponent(float amax)
{
    if (!(amax > 0.f))
        return 0;
    int e;
    frexpf(amax, &e);
    return 7 - e;
}

// Split eight scaled activations y[p] into three E4M3 limbs, exactly:
// hi = rne8(y), mid = rne8(y - hi), lo = rne8(y - hi - mid).  Each limb is
// returned as two 32-bit words (bytes in element order).
struct Limbs {
    uint32_t hi[2], mid[2], lo[2];
};

__device__ __forceinline__ void pack8_fp8(const float *v, uint32_t *out)
{
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        int w = __builtin_amdgcn_cvt_pk_fp8_f32(v[4 * h + 0], v[4 * h + 1], 0, false);
        w = __builtin_amdgcn_cvt_pk_fp8_f32(v[4 * h + 2], v[4 * h + 3], w, true);
        out[h] = (uint32_t)w;
    }
}

__device__ __forceinline__ void sub_fp8(float *v, const uint32_t *q)
{
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        const int w = (int)q[p / 4];
        float b;
        switch (p % 4) {
        case 0: b = __builtin_amdgcn_cvt_f32_fp8(w, 0); break;
        case 1: b = __builtin_amdgcn_cvt_f32_fp8(w, 1); break;
        case 2: b = __builtin_amdgcn_cvt_f32_fp8(w, 2); break;
        default: b = __builtin_amdgcn_cvt_f32_fp8(w, 3); break;
        }
        v[p] -= b;
    }
}

__device__ __forceinline__ Limbs make_limbs(uint4 xv, float scale)
{
    float y[8];
    const uint32_t w[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        y[2 * i] = half_bits_to_float(w[i] & 0xffffu) * scale;
        y[2 * i + 1] = half_bits_to_float(w[i] >> 16) * scale;
    }
    Limbs L;
    pack8_fp8(y, L.hi);
    sub_fp8(y, L.hi);
    pack8_fp8(y, L.mid);
    sub_fp8(y, L.mid);
    pack8_fp8(y, L.lo);
    return L;
}

__device__ __forceinline__ v4f mfma_fp4_fp8(const v8i &a, const v8i &b, const v4f &c)
{
    // A: fp4 E2M1 (cbsz = 4), B: fp8 E4M3 (blgp = 0), unit E8M0 scales (127).
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 4, 0, 0, 127, 0, 127);
}

__device__ __forceinline__ v8i lds_operand(const unsigned char *lo, const unsigned char *hi)
{
    const uint4 l = *(const uint4 *)lo;
    const uint4 h = *(const uint4 *)hi;
    v8i r;
    r[0] = (int)l.x;
    r[1] = (int)l.y;
    r[2] = (int)l.z;
    r[3] = (int)l.w;
    r[4] = (int)h.x;
    r[5] = (int)h.y;
    r[6] = (int)h.z;
    r[7] = (int)h.w;
    return r;
}

// k coefficients of one (row, group) from a device coefficient block, as raw
// binary16 words (c0 | c1 << 16, c2 | c3 << 16); planes >= k read as zero.
__device__ __forceinline__ uint2 load_coeffs(const uint16_t *p, int k)
{
    if (k == 4)
        return *(const uint2 *)p;
    uint2 r = make_uint2(0u, 0u);
    if (k == 2) {
        r.x = *(const uint32_t *)p;
        return r;
    }
    r.x = p[0];
    if (k > 1)
        r.x |= (uint32_t)p[1] << 16;
    if (k > 2)
        r.y = p[2];
    return r;
}

__device__ __forceinline__ float apply_coeffs(uint2 c, const v4f &d)
{
    float s = half_bits_to_float(c.x & 0xffffu) * d[0];
    s = fmaf(half_bits_to_float(c.x >> 16), d[1], s);
    s = fmaf(half_bits_to_float(c.y & 0xffffu), d[2], s);
    s = fmaf(half_bits_to_float(c.y >> 16), d[3], s);
    return s;
}

struct GemvArgs {
    const uint4 *planes;    // device plane blocks
    const uint16_t *coeffs; // device coefficient blocks
    const uint16_t *x;      // binary16 [B][I]
    uint16_t *y;            // binary16 [B][O]
    int O, I, k, n_tiles, n_gblocks, gpw, B;
};

// --------------------------------------------------------------------------
// Batch-1 GEMV.  Grid: one workgroup per T tiles (4T rows).  Wavefront w owns
// gblocks [w*gpw, (w+1)*gpw).  LDS per wavefront: 2 KiB of activation limbs
// laid out [word q][group slot s][limb l (3 = zeros)][32 bytes, k-slot order].
// --------------------------------------------------------------------------

constexpr int B1_WAVE_LDS = 2048;

template <int T>
__global__ void __launch_bounds__(512) gemv_b1_kernel(GemvArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int nw = blockDim.x >> 6;
    unsigned char *lds = smem + wv * B1_WAVE_LDS;
    float *red = (float *)(smem + nw * B1_WAVE_LDS);

    const int k = a.k;
    const int tile0 = blockIdx.x * T;
    const int gb_begin = wv * a.gpw;
    const int gb_end = min(a.n_gblocks, gb_begin + a.gpw);

    // zero the limb-3 chunks: they feed the unused 4th column of each slot
    *(uint2 *)(lds + ((lane >> 2) * 4 + 3) * 32 + 8 * (lane & 3)) = make_uint2(0u, 0u);

    // scale from the activation range this wavefront covers
    float amax = 0.f;
    for (int gb = gb_begin; gb < gb_end; ++gb) {
        const int e = gb * (GB * GROUP) + lane * 8;
        if (e < a.I)
            amax = fmaxf(amax, absmax8(*(const uint4 *)(a.x + e)));
    }
    const int sigma = scale_exponent(wave_max(amax));
    const float lscale = ldexpf(1.0f, sigma + inv_alpha_exp(lane & 3));
    const float inv_scale = ldexpf(1.0f, -sigma);

    // limb writes: lane owns elements 8*lane .. 8*lane+7 of the gblock:
    // group slot lane/16, word (lane%16)/4, k-slots 8*(lane%4) ..
    const int wr_off = ((((lane & 15) >> 2) * 4 + (lane >> 4)) * 4) * 32 + 8 * (lane & 3);
    // B-operand reads: column n = lane%16 = (slot s, limb l), k-block lane/16
    const int n = lane & 15, kb = lane >> 4;
    const int s = n >> 2, l = n & 3;
    const bool act = (l < 3) && ((kb >> 1) == (s & 1));
    const int data_off = (s * 4 + l) * 32 + 16 * (kb & 1);
    const int zero_off = (s * 4 + 3) * 32;
    const int lo_off = (act && s < 2) ? data_off : zero_off;
    const int hi_off = (act && s >= 2) ? data_off : zero_off;
    // A operand: row m = lane%16 = (tile row r, plane i), k-block = group slot
    const int a_r = (lane & 15) >> 2, a_i = lane & 3, a_b = lane >> 4;
    const bool a_ok = a_i < k;
    const int a_slot = (a_b * TILE_ROWS + a_r) * k + a_i;
    // coefficients: D rows of this lane are tile row lane/16, planes 0..3
    const int c_entry = ((lane >> 4) * GB + ((lane & 15) >> 2)) * k;
    const size_t pblk = (size_t)GB * TILE_ROWS * k;  // uint4 per plane block
    const size_t cblk = coeff_block_entries(k);

    float acc[T];
    uint4 p_cur[T];
    uint2 c_cur[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
        acc[t] = 0.f;
        p_cur[t] = make_uint4(0u, 0u, 0u, 0u);
        c_cur[t] = make_uint2(0u, 0u);
    }
    uint4 x_cur = make_uint4(0u, 0u, 0u, 0u);

    auto fetch = [&](int gb, uint4 *p, uint2 *c, uint4 &xv) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const int tile = tile0 + t;
            if (tile < a.n_tiles) {
                const size_t blk = (size_t)tile * a.n_gblocks + gb;
                p[t] = a_ok ? a.planes[blk * pblk + a_slot] : make_uint4(0u, 0u, 0u, 0u);
                c[t] = load_coeffs(a.coeffs + blk * cblk + c_entry, k);
            } else {
                p[t] = make_uint4(0u, 0u, 0u, 0u);
                c[t] = make_uint2(0u, 0u);
            }
        }
        const int e = gb * (GB * GROUP) + lane * 8;
        xv = (e < a.I) ? *(const uint4 *)(a.x + e) : make_uint4(0u, 0u, 0u, 0u);
    };

    if (gb_begin < gb_end)
        fetch(gb_begin, p_cur, c_cur, x_cur);

    for (int gb = gb_begin; gb < gb_end; ++gb) {
        uint4 p_nxt[T];
        uint2 c_nxt[T];
        uint4 x_nxt = make_uint4(0u, 0u, 0u, 0u);
        const bool more = gb + 1 < gb_end;
        if (more)
            fetch(gb + 1, p_nxt, c_nxt, x_nxt);

        // activation limbs of this gblock -> LDS -> block-diagonal B operands
        const Limbs L = make_limbs(x_cur, lscale);
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
            d = mfma_fp4_fp8(fp4_operand(p_cur[t].x), Bq[0], d);
            d = mfma_fp4_fp8(fp4_operand(p_cur[t].y), Bq[1], d);
            d = mfma_fp4_fp8(fp4_operand(p_cur[t].z), Bq[2], d);
            d = mfma_fp4_fp8(fp4_operand(p_cur[t].w), Bq[3], d);
            acc[t] += apply_coeffs(c_cur[t], d);
        }
        if (more) {
#pragma unroll
            for (int t = 0; t < T; ++t) {
                p_cur[t] = p_nxt[t];
                c_cur[t] = c_nxt[t];
            }
            x_cur = x_nxt;
        }
    }

    // sum the 16 columns (group slot x limb) of each row, then the wavefronts
#pragma unroll
    for (int t = 0; t < T; ++t) {
        float v = acc[t] * inv_scale;
        v += __shfl_xor(v, 8);
        v += __shfl_xor(v, 4);
        v += __shfl_xor(v, 2);
        v += __shfl_xor(v, 1);
        if ((lane & 15) == 0)
            red[(wv * T + t) * TILE_ROWS + (lane >> 4)] = v;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < T * TILE_ROWS; idx += blockDim.x) {
        const int t = idx / TILE_ROWS, r = idx % TILE_ROWS;
        const int o = (tile0 + t) * TILE_ROWS + r;
        if (o < a.O) {
            float v = 0.f;
            for (int w = 0; w < nw; ++w)
                v += red[(w * T + t) * TILE_ROWS + r];
            a.y[o] = __half_as_ushort(__float2half_rn(v));
        }
    }
}

// --------------------------------------------------------------------------
// Small-batch GEMM (B <= 8).  One instruction per (tile, group, column set);
// columns are (vector, limb) with five vectors per set.  LDS per wavefront:
// limbs [group slot][vector][limb][128 bytes, element order] + 16 zero bytes.
// --------------------------------------------------------------------------

constexpr int SB_VEC_PER_SET = 5;

__host__ __device__ constexpr int sb_wave_lds(int B) { return GB * B * 3 * GROUP + 16; }

template <int T, int NS>
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

    const int k = a.k;
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
                const uint2 c = load_coeffs(cb + gs * k, k);
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

// --------------------------------------------------------------------------
// Host side: validation, launch configuration.
// --------------------------------------------------------------------------

static bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

static int check_shape(int O, int I, int k)
{
    if (O < 1 || I < GROUP || I % GROUP != 0 || k < 1)
        return SBVR_E_INVALID_ARG;
    if (k > MAX_K)
        return SBVR_E_UNSUPPORTED;
    // element offsets are held in 32-bit ints
    if ((long long)O * I > (1ll << 31) - 1 || (long long)I > (1ll << 28))
        return SBVR_E_UNSUPPORTED;
    return SBVR_OK;
}

struct LaunchCfg {
    int T, gpw, waves;
};

// Rows per workgroup: 16 (4 tiles) when that still gives >= one workgroup per
// CU (256 CUs), fewer otherwise.  Each wavefront takes 1, 2 or 4 gblocks
// (512 inner elements each), more for very long rows; at most 8 wavefronts
// per workgroup.
static LaunchCfg choose_b1(const Dims &d)
{
    LaunchCfg c;
    c.T = (d.n_tiles >= 4 * 256) ? 4 : (d.n_tiles >= 2 * 256 ? 2 : 1);
    int gpw = d.n_gblocks <= 8 ? 1 : (d.n_gblocks <= 32 ? 2 : 4);
    const int min_gpw = (d.n_gblocks + 7) / 8;
    if (gpw < min_gpw)
        gpw = min_gpw;
    c.gpw = gpw;
    c.waves = (d.n_gblocks + gpw - 1) / gpw;
    return c;
}

// Small batch: the per-wavefront limb buffer grows with B, so the number of
// wavefronts per workgroup is capped to keep dynamic LDS within 64 KiB.
static size_t sb_red_bytes_per_wave(int T, int ns) { return (size_t)T * ns * TILE_ROWS * 16 * 4; }

static LaunchCfg choose_sb(const Dims &d, int B)
{
    LaunchCfg c;
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

static int launch(const void *fn, dim3 grid, dim3 block, size_t lds, hipStream_t stream, void **args)
{
    return hipLaunchKernel(fn, grid, block, args, lds, stream) == hipSuccess ? SBVR_OK : SBVR_E_HIP;
}

static int launch_b1(const Dims &d, const GemvArgs &a0, hipStream_t stream)
{
    const LaunchCfg c = choose_b1(d);
    GemvArgs a = a0;
    a.gpw = c.gpw;
    const int grid = (d.n_tiles + c.T - 1) / c.T;
    const size_t lds = (size_t)c.waves * B1_WAVE_LDS + (size_t)c.waves * c.T * TILE_ROWS * 4;
    const dim3 block(64 * c.waves);
    void *args[] = {&a};
    const void *fn = c.T == 4 ? (const void *)gemv_b1_kernel<4>
                   : c.T == 2 ? (const void *)gemv_b1_kernel<2>
                              : (const void *)gemv_b1_kernel<1>;
    return launch(fn, dim3(grid), block, lds, stream, args);
}

static int launch_sb(const Dims &d, const GemvArgs &a0, hipStream_t stream)
{
    const LaunchCfg c = choose_sb(d, a0.B);
    GemvArgs a = a0;
    a.gpw = c.gpw;
    const int ns = (a.B + SB_VEC_PER_SET - 1) / SB_VEC_PER_SET;
    const int grid = (d.n_tiles + c.T - 1) / c.T;
    const size_t lds = (size_t)c.waves * (sb_wave_lds(a.B) + sb_red_bytes_per_wave(c.T, ns));
    const dim3 block(64 * c.waves);
    void *args[] = {&a};
    const void *fn = c.T == 2 ? (ns == 1 ? (const void *)gemm_sb_kernel<2, 1> : (const void *)gemm_sb_kernel<2, 2>)
                              : (ns == 1 ? (const void *)gemm_sb_kernel<1, 1> : (const void *)gemm_sb_kernel<1, 2>);
    return launch(fn, dim3(grid), block, lds, stream, args);
}

}  // namespace sbvr

using namespace sbvr;

extern "C" {

const char *sbvr_status_string(int status)
{
    switch (status) {
    case SBVR_OK: return "SBVR_OK";
    case SBVR_E_INVALID_ARG: return "SBVR_E_INVALID_ARG";
    case SBVR_E_UNSUPPORTED: return "SBVR_E_UNSUPPORTED";
    case SBVR_E_WORKSPACE: return "SBVR_E_WORKSPACE";
    case SBVR_E_ALIGNMENT: return "SBVR_E_ALIGNMENT";
    case SBVR_E_HIP: return "SBVR_E_HIP";
    default: return "SBVR_E_UNKNOWN";
    }
}

int sbvr_version(void) { return 100; }

size_t sbvr_packed_plane_bytes(int O, int I, int k)
{
    if (check_shape(O, I, k) != SBVR_OK)
        return 0;
    return plane_bytes(make_dims(O, I, k));
}

size_t sbvr_packed_coeff_bytes(int O, int I, int k)
{
    if (check_shape(O, I, k) != SBVR_OK)
        return 0;
    return coeff_bytes(make_dims(O, I, k));
}

size_t sbvr_workspace_bytes(int O, int I, int k, int B)
{
    (void)O;
    (void)I;
    (void)k;
    (void)B;
    return 0;
}

static unsigned grid_for(size_t total) { return (unsigned)((total + 255) / 256); }

int sbvr_pack(int O, int I, int k, const uint32_t *planes_canon, const uint16_t *coeffs_canon,
              void *planes_dev, void *coeffs_dev, hipStream_t stream)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if (!planes_canon || !coeffs_canon || !planes_dev || !coeffs_dev)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_canon, 16) || !aligned(coeffs_canon, 2) || !aligned(planes_dev, 16) ||
        !aligned(coeffs_dev, 16))
        return SBVR_E_ALIGNMENT;
    Dims d = make_dims(O, I, k);
    size_t pw = plane_bytes(d) / 4, ce = coeff_bytes(d) / 2;
    uint32_t *pd = (uint32_t *)planes_dev;
    uint16_t *cd = (uint16_t *)coeffs_dev;
    void *pargs[] = {&d, &planes_canon, &pd, &pw};
    st = launch((const void *)pack_planes_kernel, dim3(grid_for(pw)), dim3(256), 0, stream, pargs);
    if (st != SBVR_OK)
        return st;
    void *cargs[] = {&d, &coeffs_canon, &cd, &ce};
    return launch((const void *)pack_coeffs_kernel, dim3(grid_for(ce)), dim3(256), 0, stream, cargs);
}

int sbvr_unpack(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                uint32_t *planes_canon, uint16_t *coeffs_canon, hipStream_t stream)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if (!planes_canon || !coeffs_canon || !planes_dev || !coeffs_dev)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_canon, 16) || !aligned(coeffs_canon, 2) || !aligned(planes_dev, 16) ||
        !aligned(coeffs_dev, 16))
        return SBVR_E_ALIGNMENT;
    Dims d = make_dims(O, I, k);
    size_t pw = (size_t)O * d.G * k * 4, ce = (size_t)O * d.G * k;
    const uint32_t *pd = (const uint32_t *)planes_dev;
    const uint16_t *cd = (const uint16_t *)coeffs_dev;
    void *pargs[] = {&d, &pd, &planes_canon, &pw};
    st = launch((const void *)unpack_planes_kernel, dim3(grid_for(pw)), dim3(256), 0, stream, pargs);
    if (st != SBVR_OK)
        return st;
    void *cargs[] = {&d, &cd, &coeffs_canon, &ce};
    return launch((const void *)unpack_coeffs_kernel, dim3(grid_for(ce)), dim3(256), 0, stream, cargs);
}

static int check_gemv_args(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                           const uint16_t *x, const uint16_t *y, int B, size_t ws_bytes)
{
    int st = check_shape(O, I, k);
    if (st != SBVR_OK)
        return st;
    if (B < 1 || B > 8)
        return SBVR_E_INVALID_ARG;
    if (!planes_dev || !coeffs_dev || !x || !y)
        return SBVR_E_INVALID_ARG;
    if (!aligned(planes_dev, 16) || !aligned(coeffs_dev, 16) || !aligned(x, 16) || !aligned(y, 2))
        return SBVR_E_ALIGNMENT;
    if (ws_bytes < sbvr_workspace_bytes(O, I, k, B))
        return SBVR_E_WORKSPACE;
    return SBVR_OK;
}

int sbvr_gemv(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
              const uint16_t *x, uint16_t *y, void *workspace, size_t ws_bytes, hipStream_t stream)
{
    (void)workspace;
    int st = check_gemv_args(O, I, k, planes_dev, coeffs_dev, x, y, 1, ws_bytes);
    if (st != SBVR_OK)
        return st;
    const Dims d = make_dims(O, I, k);
    GemvArgs a = {(const uint4 *)planes_dev, (const uint16_t *)coeffs_dev, x, y, O, I, k,
                  d.n_tiles, d.n_gblocks, 1, 1};
    return launch_b1(d, a, stream);
}

int sbvr_gemm_small_batch(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                          const uint16_t *X, uint16_t *Y, int B, void *workspace, size_t ws_bytes,
                          hipStream_t stream)
{
    (void)workspace;
    int st = check_gemv_args(O, I, k, planes_dev, coeffs_dev, X, Y, B, ws_bytes);
    if (st != SBVR_OK)
        return st;
    const Dims d = make_dims(O, I, k);
    GemvArgs a = {(const uint4 *)planes_dev, (const uint16_t *)coeffs_dev, X, Y, O, I, k,
                  d.n_tiles, d.n_gblocks, 1, B};
    return launch_sb(d, a, stream);
}

}  // extern "C"
