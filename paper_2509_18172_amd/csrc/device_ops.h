// Device-side building blocks of the SBVR GEMV kernels for gfx950.
//
// The per-plane masked sums of Sec. 4.4 (S = sum of x over the set bits of a
// plane) are a bit-matrix times vector product.  Here it runs on the matrix
// cores as an fp4 x fp8 product:
//
//   * A operand (weights): each 32-bit device plane word w becomes four fp4
//     (E2M1) registers by masking: register v keeps bit v of every nibble, so
//     nibble p holds element 8v+p of the word as 0 or alpha_v with
//     alpha = (0.5, 1, 2, 2) (bit 3, the fp4 sign, is shifted down to bit 2).
//     No per-element work is done on the bits.
//   * B operand (binary16 activations): each activation, scaled by a power of
//     two 2^sigma / alpha_v, is split exactly into four E5M2 limbs, each the
//     top byte of a binary16 piece with at most three significant bits
//     (E5M2 is binary16 with the mantissa cut to two bits: same exponent
//     range, so no conversion instruction is needed), and
//     alpha_v * (l0 + l1 + l2 + l3) = 2^sigma * x.  With SBVR-8 activations
//     (the W4A8 path) the operand holds the 8-bit code split into two E4M3
//     limbs instead.
//   * v_mfma_scale_f32_16x16x128_f8f6f4 with unit scales multiplies and sums
//     128 k-slots per row in fp32.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>

#include "layout.h"

namespace sbvr {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

// fp4 A operand of one device plane word (registers 4..7 unused by fp4).
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

// log2(1 / alpha_v) for the elements of register v = (element in word) / 8.
__device__ __forceinline__ int inv_alpha_exp(int v) { return v == 0 ? 1 : (v == 1 ? 0 : -1); }

__device__ __forceinline__ float half_bits_to_float(uint32_t bits16)
{
    return __half2float(__ushort_as_half((unsigned short)bits16));
}

// DPP lane exchange within rows of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
constexpr int DPP_QUAD_XOR1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int DPP_QUAD_XOR2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int DPP_ROW_HALF_MIRROR = 0x141;
constexpr int DPP_ROW_MIRROR = 0x140;

// Sum over each row of 16 lanes; every lane of the row gets the row sum,
// always added in the same order for a given lane.
__device__ __forceinline__ float row16_sum(float v)
{
    v += dpp_f32<DPP_QUAD_XOR1>(v);
    v += dpp_f32<DPP_QUAD_XOR2>(v);
    v += dpp_f32<DPP_ROW_HALF_MIRROR>(v);
    v += dpp_f32<DPP_ROW_MIRROR>(v);
    return v;
}

// Wavefront index within the workgroup as a scalar (uniform) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Power-of-two exponent sigma with max|x| * 2^sigma in [2^13, 2^14): the
// scaled activations times 1/alpha (<= 2) stay below 2^15, inside both the
// binary16 and the E5M2 range (largest finite E5M2 value 57344).  sigma is
// capped at 29: a block whose maximum is below 2^-16 holds only binary16
// subnormals, multiples of 2^-24, which 2^28 already lifts to multiples of
// 2^4 (exact in the split below).  A zero block gets sigma = 0.
__device__ __forceinline__ int scale_exponent(float amax)
{
    if (!(amax > 0.f))
        return 0;
    int e;
    frexpf(amax, &e);
    return min(14 - e, 29);
}

// Four 8-bit limbs of eight activations, two words each (bytes in element
// order); limb j feeds the result column of limb j.
struct Limbs {
    uint32_t l[4][2];
};

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t h2_sub(uint32_t a, uint32_t b)
{
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(h2_t, a) - __builtin_bit_cast(h2_t, b));
}

__device__ __forceinline__ uint32_t h2_mul(uint32_t a, uint32_t f)
{
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(h2_t, a) * __builtin_bit_cast(h2_t, f));
}

// binary16 2^e in both halves, -14 <= e <= 15
__device__ __forceinline__ uint32_t h2_pow2(int e)
{
    const uint32_t b = (uint32_t)(e + 15) << 10;
    return b | (b << 16);
}

// Exact split of eight binary16 activations into four E5M2 limbs.
//
// x' = x * 2^(sigma + inv_alpha) is formed in binary16 as two exact
// power-of-two products, 2^(min(sigma, 14) + inv_alpha) and then
// 2^(sigma - min(sigma, 14)) <= 2^15 (no branch); the block maximum lands in
// [2^12, 2^15) (or below, all of it exact, for blocks of subnormals).
// The truncation split p0 = x' with its mantissa cut to two bits,
// p1 = the same cut of x' - p0, p2 = the cut of x' - p0 - p1 and
// p3 = x' - p0 - p1 - p2 is exact in binary16 (each difference is a multiple
// of x''s unit in the last place, below the piece it is taken from), and
// every piece whose bits lie at or above 2^-16 has its low byte zero: its top
// byte is then the E5M2 encoding of the same value (E5M2 = sign, the five
// binary16 exponent bits, the top two mantissa bits).  So
// x' = p0 + p1 + p2 + p3 exactly whenever x' is at least 2^-6 (its 11
// significant bits stay at or above 2^-16): for every element of at least
// 2^-18 of its block's largest magnitude.  Smaller elements lose only bits
// below 2^-16 in x' units, less than 2^-27 of the block maximum.
// sigma: the block's scale exponent (scale_exponent, wavefront-uniform);
// inv_alpha: log2(1/alpha) of the lane's elements.
__device__ __forceinline__ Limbs split_limbs(uint4 xv, int sigma, int inv_alpha)
{
    constexpr uint32_t CUT = 0xFF00FF00u;  // sign, exponent and 2 mantissa bits of each half
    const int s0 = min(sigma, 14);
    const uint32_t f = h2_pow2(s0 + inv_alpha), g = h2_pow2(sigma - s0);
    uint32_t w[4] = {h2_mul(h2_mul(xv.x, f), g), h2_mul(h2_mul(xv.y, f), g), h2_mul(h2_mul(xv.z, f), g),
                     h2_mul(h2_mul(xv.w, f), g)};
    uint32_t p[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t r = w[i];
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            p[j][i] = r & CUT;
            r = h2_sub(r, p[j][i]);
        }
        p[3][i] = r;
    }
    Limbs L;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h)  // top bytes of the four halves of two words
            L.l[j][h] = __builtin_amdgcn_perm(p[j][2 * h + 1], p[j][2 * h], 0x07050301u);
    return L;
}

__device__ __forceinline__ void pack8_fp8(const float *v, uint32_t *out)
{
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        int w = __builtin_amdgcn_cvt_pk_fp8_f32(v[4 * h + 0], v[4 * h + 1], 0, false);
        w = __builtin_amdgcn_cvt_pk_fp8_f32(v[4 * h + 2], v[4 * h + 3], w, true);
        out[h] = (uint32_t)w;
    }
}

// Online conversion to SBVR-8 activations (Sec. 4.3, Eq. 12) for the W4A8
// decode path.  The lanes 16r .. 16r+15 of a wavefront hold the 128 elements
// of group r of the gblock (eight each).  Per group: s = absmax / 127 and the
// 8-bit code q = rne(fl(x / s)) within +-127 (binary32, correctly rounded
// division; a zero group has s = 0, q = 0).  Eq. 12's coefficients are the
// two's-complement weights of q, so the matrix-core operand carries q itself,
// split exactly into two E4M3 limbs: 16 * floor(q / 16) and q mod 16 (each
// divided by alpha_v, still exact), in limb slots 0 and 1 (2 and 3 are zero).
// Returns the limbs; `out_scale` receives the scale of the group of the
// lane's result column (slot (lane % 16) / 4), which multiplies its sums.
//
// The code is taken from t = x * rcp(s) when t is clearly away from a
// half-integer: rcp is within 1 ulp and the product adds half an ulp, so
// |t - fl(x / s)| <= 2^-22 |x / s| <= 2^-15 (|x / s| <= 128); a distance of
// at least 2^-14 from the nearest half-integer then gives the same rounded
// integer as fl(x / s).  Elements closer than that (rare) use the correctly
// rounded division.
__device__ __forceinline__ float row16_max(float v)
{
    v = fmaxf(v, dpp_f32<DPP_QUAD_XOR1>(v));
    v = fmaxf(v, dpp_f32<DPP_QUAD_XOR2>(v));
    v = fmaxf(v, dpp_f32<DPP_ROW_HALF_MIRROR>(v));
    v = fmaxf(v, dpp_f32<DPP_ROW_MIRROR>(v));
    return v;
}

__device__ __forceinline__ Limbs a8_limbs(uint4 xv, int lane, int inv_alpha, float &out_scale)
{
    const uint32_t w[4] = {xv.x, xv.y, xv.z, xv.w};
    float xf[8];
    float amax = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        xf[2 * i] = half_bits_to_float(w[i] & 0xffffu);
        xf[2 * i + 1] = half_bits_to_float(w[i] >> 16);
        amax = fmaxf(amax, fmaxf(fabsf(xf[2 * i]), fabsf(xf[2 * i + 1])));
    }
    const float sg = __fdiv_rn(row16_max(amax), 127.0f);  // this lane's group
    const float r = sg > 0.f ? __builtin_amdgcn_rcpf(sg) : 0.f;
    float qf[8];
    float dmax = 0.f;  // largest |t - rint(t)| (exact differences)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float t = xf[e] * r;
        qf[e] = rintf(t);
        dmax = fmaxf(dmax, fabsf(t - qf[e]));
    }
    if (dmax >= 0.5f - 0x1p-14f) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
            qf[e] = rintf(__fdiv_rn(xf[e], sg));  // sg > 0 here: t = 0 otherwise
    }
    const float f = ldexpf(1.0f, inv_alpha), f16 = 16.0f * f;
    float hi[8], lo[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float q = fminf(127.f, fmaxf(-127.f, qf[e]));
        const float fl = floorf(q * 0.0625f);  // floor(q / 16), exact
        hi[e] = fl * f16;
        lo[e] = fmaf(fl, -16.0f, q) * f;  // q mod 16, exact
    }
    Limbs L;
    pack8_fp8(hi, L.l[0]);
    pack8_fp8(lo, L.l[1]);
    L.l[2][0] = L.l[2][1] = L.l[3][0] = L.l[3][1] = 0u;
    const int slot = (lane & 15) >> 2;
    const float s0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sg), 0));
    const float s1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sg), 16));
    const float s2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sg), 32));
    const float s3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sg), 48));
    out_scale = slot == 0 ? s0 : (slot == 1 ? s1 : (slot == 2 ? s2 : s3));
    return L;
}

// max |x| over the wavefront's binary16 activations (eight per lane), as a
// float: the magnitudes' bit patterns order like unsigned integers.
__device__ __forceinline__ float wave_absmax_h(uint4 v)
{
    typedef unsigned short u2_t __attribute__((ext_vector_type(2)));
    const u2_t a = __builtin_bit_cast(u2_t, v.x & 0x7fff7fffu), b = __builtin_bit_cast(u2_t, v.y & 0x7fff7fffu);
    const u2_t c = __builtin_bit_cast(u2_t, v.z & 0x7fff7fffu), d = __builtin_bit_cast(u2_t, v.w & 0x7fff7fffu);
    const u2_t m2 = __builtin_elementwise_max(__builtin_elementwise_max(a, b), __builtin_elementwise_max(c, d));
    int m = (int)(m2[0] > m2[1] ? m2[0] : m2[1]);
    m = max(m, __builtin_amdgcn_update_dpp(0, m, DPP_QUAD_XOR1, 0xf, 0xf, false));
    m = max(m, __builtin_amdgcn_update_dpp(0, m, DPP_QUAD_XOR2, 0xf, 0xf, false));
    m = max(m, __builtin_amdgcn_update_dpp(0, m, DPP_ROW_HALF_MIRROR, 0xf, 0xf, false));
    m = max(m, __builtin_amdgcn_update_dpp(0, m, DPP_ROW_MIRROR, 0xf, 0xf, false));
    const int r = max(max(__builtin_amdgcn_readlane(m, 0), __builtin_amdgcn_readlane(m, 16)),
                      max(__builtin_amdgcn_readlane(m, 32), __builtin_amdgcn_readlane(m, 48)));
    return half_bits_to_float((uint32_t)r);
}

// 4 x 4 transpose of 32-bit words across the lanes l, l+16, l+32, l+48 of a
// wavefront: lane l + 16 b holds words (w[b][0], ..., w[b][3]) on entry and
// (w[0][b], ..., w[3][b]) on exit.  permlane32_swap exchanges the upper half
// of its first operand with the lower half of its second; permlane16_swap
// does the same between odd and even rows of 16 lanes.
__device__ __forceinline__ uint4 transpose_rows4(uint4 w)
{
    const auto s02 = __builtin_amdgcn_permlane32_swap(w.x, w.z, false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(w.y, w.w, false, false);
    const auto t01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
    const auto t23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
    return make_uint4(t01[0], t01[1], t23[0], t23[1]);
}

// A: fp4 E2M1 (cbsz = 4); B: E5M2 (blgp = 1) for binary16 activations, E4M3
// (blgp = 0) for the SBVR-8 codes; unit E8M0 scales (127).
template <bool A8>
__device__ __forceinline__ v4f mfma_fp4_fp8(const v8i &a, const v8i &b, const v4f &c)
{
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 4, A8 ? 0 : 1, 0, 127, 0, 127);
}

// An 8-register fp8 B operand from two 16-byte LDS chunks (k-slot halves).
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

// Weight loads: 16-byte plane slots and coefficient words are streamed once,
// so they are loaded non-temporally (no reuse expected in the caches).
typedef unsigned v4u_t __attribute__((ext_vector_type(4)));
typedef unsigned v2u_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint4 load_nt16(const uint4 *p)
{
    const v4u_t v = __builtin_nontemporal_load((const v4u_t *)p);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

// Coefficients of a lane's four D rows.  A lane of a 16x16 result holds the
// rows m = 4q .. 4q+3 (q = lane / 16) of one column; for one group slot b
// their coefficients are the contiguous entries (q * GB + b) * CPL + j of the
// coefficient block (j < CPL = 4 coefficients, 3 for K = 3), returned as raw
// binary16 words (c0 | c1 << 16, c2 | c3 << 16); missing ones read zero.
template <int K>
__host__ __device__ constexpr int coefs_per_lane() { return coefs_per_quad(K); }

template <int K>
__device__ __forceinline__ uint2 load_coefs4(const uint16_t *p)
{
    if constexpr (K == 3) {
        return make_uint2((uint32_t)p[0] | ((uint32_t)p[1] << 16), (uint32_t)p[2]);
    } else {
        const v2u_t v = __builtin_nontemporal_load((const v2u_t *)p);
        return make_uint2(v[0], v[1]);
    }
}

// Row partial sums of a lane: the coefficients times its four D values,
// grouped by output row.  A rows m = r * RS + i (RS = row slots), so a lane's
// four rows belong to NP = 4 / RS tile rows: rows q * NP + p, p < NP.
template <int K>
__host__ __device__ constexpr int partials_per_lane() { return 4 / row_slots(K); }

template <int K>
__device__ __forceinline__ void apply_coefs(uint2 c, const v4f &d, float *p)
{
    const float c0 = half_bits_to_float(c.x & 0xffffu), c1 = half_bits_to_float(c.x >> 16);
    const float c2 = half_bits_to_float(c.y & 0xffffu), c3 = half_bits_to_float(c.y >> 16);
    if constexpr (row_slots(K) == 4) {
        p[0] = fmaf(c3, d[3], fmaf(c2, d[2], fmaf(c1, d[1], c0 * d[0])));
    } else if constexpr (row_slots(K) == 2) {
        p[0] = fmaf(c1, d[1], c0 * d[0]);
        p[1] = fmaf(c3, d[3], c2 * d[2]);
    } else {
        p[0] = c0 * d[0];
        p[1] = c1 * d[1];
        p[2] = c2 * d[2];
        p[3] = c3 * d[3];
    }
}

// A-operand slot of a lane within a plane block: lane (row m = lane % 16,
// k-block b = lane / 16) takes the 16 bytes of (group slot b, tile row
// m / RS, plane m % RS); `ok` is false for the empty plane slots of K = 3.
template <int K>
__device__ __forceinline__ unsigned a_slot_bytes(int lane, bool &ok)
{
    constexpr int RS = row_slots(K), TR = tile_rows(K);
    const int m = lane & 15, b = lane >> 4;
    const int r = m / RS, i = m % RS;
    ok = i < K;
    return (unsigned)((b * TR + r) * K + (ok ? i : 0)) * 16u;
}

// Buffer-resource loads.  A descriptor bounds a byte range; a lane whose
// offset falls outside it reads zero and issues no memory access, which lets
// a software pipeline prefetch past the end of its range unconditionally.
typedef __amdgpu_buffer_rsrc_t buf_rsrc;
constexpr unsigned BUF_DWORD3 = 0x00020000u;  // raw (untyped) buffer, gfx9 family
constexpr int BUF_NT = 2;                     // non-temporal cache policy
constexpr unsigned BUF_OOB = 0x80000000u;     // an offset beyond every range used here
constexpr unsigned LANE_OOB = 0x40000000u;    // per-lane offset that reads zero (the host caps ranges below 2^30)

__device__ __forceinline__ buf_rsrc make_rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, BUF_DWORD3);
}

__device__ __forceinline__ uint4 buf_load16(buf_rsrc r, unsigned off)
{
    const v4u_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, BUF_NT);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

// load_coefs4 through a descriptor (byte offset of the lane's first entry).
template <int K>
__device__ __forceinline__ uint2 buf_coefs4(buf_rsrc r, unsigned off)
{
    if constexpr (K == 3) {
        const unsigned c0 = __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, BUF_NT);
        const unsigned c1 = __builtin_amdgcn_raw_buffer_load_b16(r, off + 2, 0, BUF_NT);
        const unsigned c2 = __builtin_amdgcn_raw_buffer_load_b16(r, off + 4, 0, BUF_NT);
        return make_uint2(c0 | (c1 << 16), c2);
    } else {
        const v2u_t v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, BUF_NT);
        return make_uint2(v[0], v[1]);
    }
}

// Coefficient-cache format: a lane's NP = TR / 4 index entries (NP = 1, 2:
// one dword; NP = 4: two) and the gather of its four D rows' coefficients
// from the cache (TABLE_STRIDE entries per set).  The cache is read through a
// descriptor bounded by the number of sets: an index past the end reads zero
// coefficients instead of faulting.
template <int K>
struct IxLane {
    typedef typename std::conditional<(index_per_lane(K) == 4), uint2, uint32_t>::type type;
};

template <int K>
__device__ __forceinline__ typename IxLane<K>::type buf_index(buf_rsrc r, unsigned off)
{
    if constexpr (index_per_lane(K) == 4) {
        const v2u_t v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, BUF_NT);
        return make_uint2(v[0], v[1]);
    } else if constexpr (index_per_lane(K) == 2) {
        return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, BUF_NT);
    } else {
        return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, BUF_NT);
    }
}

template <int K>
__device__ __forceinline__ uint2 table_coefs4(buf_rsrc t, typename IxLane<K>::type ix)
{
    constexpr unsigned SET_B = TABLE_STRIDE * 2;
    if constexpr (index_per_lane(K) == 4) {  // four rows, plane 0 of each
        const unsigned c0 = __builtin_amdgcn_raw_buffer_load_b16(t, (ix.x & 0xffffu) * SET_B, 0, 0);
        const unsigned c1 = __builtin_amdgcn_raw_buffer_load_b16(t, (ix.x >> 16) * SET_B, 0, 0);
        const unsigned c2 = __builtin_amdgcn_raw_buffer_load_b16(t, (ix.y & 0xffffu) * SET_B, 0, 0);
        const unsigned c3 = __builtin_amdgcn_raw_buffer_load_b16(t, (ix.y >> 16) * SET_B, 0, 0);
        return make_uint2(c0 | (c1 << 16), c2 | (c3 << 16));
    } else if constexpr (index_per_lane(K) == 2) {  // two rows, planes 0 and 1
        const unsigned v0 = __builtin_amdgcn_raw_buffer_load_b32(t, (ix & 0xffffu) * SET_B, 0, 0);
        const unsigned v1 = __builtin_amdgcn_raw_buffer_load_b32(t, (ix >> 16) * SET_B, 0, 0);
        return make_uint2(v0, v1);
    } else {  // one row, planes 0..3 (plane 3 of K = 3 is the zero padding)
        const v2u_t v = __builtin_amdgcn_raw_buffer_load_b64(t, ix * SET_B, 0, 0);
        return make_uint2(v[0], v[1]);
    }
}

struct GemvArgs {
    const uint4 *planes;    // device plane blocks
    const uint16_t *coeffs; // device coefficient blocks (per-group format)
    const uint16_t *x;      // binary16 [B][I]
    uint16_t *y;            // binary16 [B][O]
    int O, I, k, n_tiles, n_gblocks, gpw, B;
    int tpw;                // tiles per workgroup (streaming kernel)
    const uint16_t *index;  // device index blocks (coefficient-cache format)
    const uint16_t *table;  // coefficient sets [n_sets][TABLE_STRIDE]
    int n_sets;
};

// Grouped launch: several GEMVs with the same inner dimension and plane count
// (each with its own weights, activations and output) in one dispatch.
// Member m owns the workgroups [wg0[m], wg0[m + 1]); entries past the last
// member hold wg0 = INT_MAX.
constexpr int GROUP_MAX = 4;
struct GemvGroup {
    const uint4 *planes[GROUP_MAX];
    const uint16_t *coeffs[GROUP_MAX];
    const uint16_t *x[GROUP_MAX];
    uint16_t *y[GROUP_MAX];
    int O[GROUP_MAX];
    int n_tiles[GROUP_MAX];
    int wg0[GROUP_MAX];
};

template <class T>
__device__ __forceinline__ T group_pick(const T (&v)[GROUP_MAX], int m)
{
    return m == 0 ? v[0] : (m == 1 ? v[1] : (m == 2 ? v[2] : v[3]));
}

// Binds `a` to the member that owns workgroup `bid` of a grouped launch and
// returns the workgroup's index within that member (all wavefront-uniform).
__device__ __forceinline__ int bind_group_member(const GemvGroup &g, GemvArgs &a, int bid)
{
    const int m = (bid >= g.wg0[1]) + (bid >= g.wg0[2]) + (bid >= g.wg0[3]);
    a.planes = group_pick(g.planes, m);
    a.coeffs = group_pick(g.coeffs, m);
    a.x = group_pick(g.x, m);
    a.y = group_pick(g.y, m);
    a.O = group_pick(g.O, m);
    a.n_tiles = group_pick(g.n_tiles, m);
    return bid - group_pick(g.wg0, m);
}

}  // namespace sbvr
