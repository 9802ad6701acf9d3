// Small-batch SBVR GEMM (2 <= B <= 8 activation vectors; Sec. 4.4 applied to
// each vector), streaming the weights once for all B vectors.
//
// Work decomposition (as the batch-1 streaming kernel): a workgroup owns tpw
// consecutive tiles (TR rows) and every gblock (512 inner elements) of them;
// wavefront w takes gblocks w, w+W, ...  Its items (gblock, tile) stream
// through a D-deep register ring loaded with buffer descriptors bounded by
// the workgroup's tile range (loads past the end read zero, no traffic).
//
// Matrix-core formulation.  One 16x16x128 fp4 x fp8 instruction per (tile,
// group, column set): the 128 k-slots are one whole group (its four plane
// words, one per 32-slot k-block), rows are (tile row, plane) and the 16
// columns are (vector, limb) with four columns per vector -- the four E5M2
// limbs of its activations -- so a column set serves four vectors (B <= 4:
// one set, B <= 8: two).  The device layout gives lane (row m, k-block b) the four
// words of group b; a 4 x 4 cross-lane transpose turns that into word b of
// the four groups, i.e. the A operands of the four instructions of an item.
//
// Each lane applies the coefficients of its four D rows (the planes of 1, 2 or
// 4 tile rows) for every group as one chain of fused multiply-adds and adds
// the item's (row, vector, limb) partial to LDS; at the end the workgroup sums,
// per output, the wavefronts in order and the four limb columns of its
// vector (deterministic, no global workspace).
#include "device_ops.h"
#include "launch.h"

namespace sbvr {

// Ring depth: 3 when a workgroup streams many tiles (long item sequences per
// wavefront), 2 otherwise (its shorter prologue wins when each wavefront has
// only a few items).
#ifndef SBVR_SBS_DEPTH_LONG
#define SBVR_SBS_DEPTH_LONG 3
#endif
#ifndef SBVR_SBS_DEPTH_SHORT
#define SBVR_SBS_DEPTH_SHORT 2
#endif
#ifndef SBVR_SBS_LONG_TPW
#define SBVR_SBS_LONG_TPW 12
#endif
// Ring depth when a wavefront takes several gblocks (long rows) at B <= 4:
// its item stream crosses gblocks, and the deeper ring keeps the next
// gblock's first items in flight while its operand is built (measured at
// B = 4: 8B down 14.0 -> 13.0 us, 70B down 40.3 -> 36.4, 70B gate/up 31.5 ->
// 30.3; B = 2: 11.3 -> 10.9, 34.0 -> 31.6, 29.5 -> 28.7; no gain at B = 8,
// where the VALU work per item bounds the kernel).
#ifndef SBVR_SBS_DEPTH_MULTI_SMALL
#define SBVR_SBS_DEPTH_MULTI_SMALL 4
#endif
#ifndef SBVR_SBS_MAX_WAVES
#define SBVR_SBS_MAX_WAVES 8
#endif
#ifndef SBVR_SBS_GROUPS
#define SBVR_SBS_GROUPS 256
#endif

// vectors per column set, and the LDS staging per wavefront: the limbs of
// two vectors at a time, [group][vector of the pair][limb][128 bytes], then
// 256 zero bytes, read by the columns of absent vectors at a different 16
// bytes per lane of a 16-lane group (a set of four vectors is staged in two
// phases, which keeps eight wavefronts' staging within 35 KB)
constexpr int SBS_VPS = 4;
// LDS a small-batch workgroup may use (of the 160 KiB of a gfx950 CU; one
// workgroup per CU runs anyway at this kernel's register use)
constexpr size_t SBS_LDS_MAX = 160 * 1024;
__host__ __device__ constexpr int sbs_sets(int nb) { return (nb + SBS_VPS - 1) / SBS_VPS; }
__host__ __device__ constexpr int sbs_vps(int nb) { return nb < SBS_VPS ? nb : SBS_VPS; }
__host__ __device__ constexpr int sbs_stage_bytes(int) { return GB * 2 * 4 * GROUP + 256; }

// max |x| over the wavefront for two activation vectors at once (eight
// binary16 values per lane each): the magnitudes' bit patterns are compared as
// 16-bit integers, vector a in the low and vector b in the high half of one
// register, reduced within each row of 16 lanes by DPP and across the rows by
// two lane swaps (the semantics transpose_rows4 relies on), so the result
// needs one read into a scalar register instead of one per row and vector.
// Returns both maxima as binary16 bit patterns (a: bits 0-15, b: bits
// 16-31), wavefront-uniform.
__device__ __forceinline__ uint32_t wave_absmax2_bits(uint4 a, uint4 b)
{
    typedef unsigned short u2_t __attribute__((ext_vector_type(2)));
    auto lane_max = [](uint4 v) {
        const u2_t p = __builtin_bit_cast(u2_t, v.x & 0x7fff7fffu), q = __builtin_bit_cast(u2_t, v.y & 0x7fff7fffu);
        const u2_t r = __builtin_bit_cast(u2_t, v.z & 0x7fff7fffu), t = __builtin_bit_cast(u2_t, v.w & 0x7fff7fffu);
        return __builtin_elementwise_max(__builtin_elementwise_max(p, q), __builtin_elementwise_max(r, t));
    };
    const u2_t ma = lane_max(a), mb = lane_max(b);
    const u2_t lo = {ma[0], mb[0]}, hi = {ma[1], mb[1]};
    uint32_t w = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(lo, hi));
    auto pmax = [](uint32_t x, uint32_t y) {
        return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u2_t, x),
                                                                      __builtin_bit_cast(u2_t, y)));
    };
    w = pmax(w, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, DPP_QUAD_XOR1, 0xf, 0xf, false));
    w = pmax(w, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, DPP_QUAD_XOR2, 0xf, 0xf, false));
    w = pmax(w, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, DPP_ROW_HALF_MIRROR, 0xf, 0xf, false));
    w = pmax(w, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, DPP_ROW_MIRROR, 0xf, 0xf, false));
    // every lane holds its row's maximum: lanes 32-63 trade with 0-31, then
    // odd rows with even rows
    const auto s32 = __builtin_amdgcn_permlane32_swap(w, w, false, false);
    w = pmax(s32[0], s32[1]);
    const auto s16 = __builtin_amdgcn_permlane16_swap(w, w, false, false);
    w = pmax(s16[0], s16[1]);
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)w);
}

// The coefficients of a lane's four D rows for the four groups of a gblock:
// 4 * CPL contiguous binary16 entries (q * GB * CPL ..), group g's at g * CPL.
template <int K>
struct CoefGroups {
    uint32_t w[2 * coefs_per_lane<K>()];
};

template <int K>
__device__ __forceinline__ CoefGroups<K> buf_coef_groups(buf_rsrc r, unsigned off)
{
    CoefGroups<K> c;
    const v4u_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, BUF_NT);
    c.w[0] = v[0];
    c.w[1] = v[1];
    c.w[2] = v[2];
    c.w[3] = v[3];
    if constexpr (coefs_per_lane<K>() == 4) {
        const v4u_t u = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16, 0, BUF_NT);
        c.w[4] = u[0];
        c.w[5] = u[1];
        c.w[6] = u[2];
        c.w[7] = u[3];
    } else {
        const v2u_t u = __builtin_amdgcn_raw_buffer_load_b64(r, off + 16, 0, BUF_NT);
        c.w[4] = u[0];
        c.w[5] = u[1];
    }
    return c;
}

// group g's coefficients as apply_coefs takes them
template <int K>
__device__ __forceinline__ uint2 coef_group(const CoefGroups<K> &c, int g)
{
    if constexpr (coefs_per_lane<K>() == 4) {
        return make_uint2(c.w[2 * g], c.w[2 * g + 1]);
    } else {
        auto h = [&](int e) { return e & 1 ? c.w[e >> 1] >> 16 : c.w[e >> 1] & 0xffffu; };
        return make_uint2(h(3 * g) | (h(3 * g + 1) << 16), h(3 * g + 2));
    }
}

// acc[p] += the coefficients times the lane's four D values of their rows
// (rows grouped by output row as in apply_coefs), one fused multiply-add per
// value with the binary16 coefficient converted on the way in
template <int K>
__device__ __forceinline__ void fma_coefs(uint2 c, const v4f &d, float *acc)
{
    const _Float16 c0 = __builtin_bit_cast(_Float16, (uint16_t)(c.x & 0xffffu));
    const _Float16 c1 = __builtin_bit_cast(_Float16, (uint16_t)(c.x >> 16));
    const _Float16 c2 = __builtin_bit_cast(_Float16, (uint16_t)(c.y & 0xffffu));
    const _Float16 c3 = __builtin_bit_cast(_Float16, (uint16_t)(c.y >> 16));
    constexpr int RS = row_slots(K);
    if constexpr (RS == 4) {
        acc[0] = fmaf((float)c0, d[0], acc[0]);
        acc[0] = fmaf((float)c1, d[1], acc[0]);
        acc[0] = fmaf((float)c2, d[2], acc[0]);
        acc[0] = fmaf((float)c3, d[3], acc[0]);
    } else if constexpr (RS == 2) {
        acc[0] = fmaf((float)c0, d[0], acc[0]);
        acc[0] = fmaf((float)c1, d[1], acc[0]);
        acc[1] = fmaf((float)c2, d[2], acc[1]);
        acc[1] = fmaf((float)c3, d[3], acc[1]);
    } else {
        acc[0] = fmaf((float)c0, d[0], acc[0]);
        acc[1] = fmaf((float)c1, d[1], acc[1]);
        acc[2] = fmaf((float)c2, d[2], acc[2]);
        acc[3] = fmaf((float)c3, d[3], acc[3]);
    }
}

template <int K, int NB, int D, bool MULTI>
__global__ void __launch_bounds__(512) gemm_sbs_kernel(GemvArgs a)
{
    constexpr int NS = sbs_sets(NB);
    constexpr int VPS = sbs_vps(NB);
    constexpr int STAGE = sbs_stage_bytes(NB);
    constexpr int ZERO0 = STAGE - 256;
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63;
    const int wv = wave_id();
    const int nw = blockDim.x >> 6;
    const int B = a.B;  // vectors actually present (<= NB)
    unsigned char *stage = smem + wv * STAGE;
    constexpr int TR = tile_rows(K), NP = partials_per_lane<K>();
    float *red = (float *)(smem + nw * STAGE);  // [tpw][nw][NS][TR rows][16 columns]

    const int tile0 = blockIdx.x * a.tpw;
    const int ntl = min(a.tpw, a.n_tiles - tile0);
    const int n_items = MULTI ? ((a.n_gblocks - wv + nw - 1) / nw) * ntl : ntl;

    // A: lane (row m = lane%16 = (tile row, plane), k-block lane/16) loads the
    // 16 bytes of group lane/16; lanes of empty plane slots (K = 3) read zero.
    bool a_ok;
    const unsigned a_slot = a_slot_bytes<K>(lane, a_ok);
    const unsigned p_lane = a_ok ? a_slot : LANE_OOB;
    // coefficients of the lane's D rows for the four group slots
    const unsigned c_lane = (unsigned)((lane >> 4) * GB * coefs_per_lane<K>()) * 2u;
    constexpr unsigned PBLK_B = GB * TR * K * 16;
    constexpr unsigned CBLK_B = GB * TR * K * 2;
    const unsigned pstep = (unsigned)a.n_gblocks * PBLK_B;
    const unsigned cstep = (unsigned)a.n_gblocks * CBLK_B;
    const size_t blk0 = (size_t)tile0 * a.n_gblocks;
    const buf_rsrc prs = make_rsrc((const unsigned char *)a.planes + blk0 * PBLK_B, (unsigned)ntl * pstep);
    const buf_rsrc crs = make_rsrc((const unsigned char *)a.coeffs + blk0 * CBLK_B, (unsigned)ntl * cstep);

    int pf_i = 0, pf_gb = wv;
    uint4 P[D];
    CoefGroups<K> C[D];
    // Slot j's planes for the next item of the stream; returns the byte
    // offset of that item's coefficients, loaded by issue_c.  The loop
    // reloads a slot's coefficients only after the item's last use of its old
    // ones: loading them with the planes kept both sets live, and the compiler
    // then rotated the ring through register copies at every loop latch,
    // behind a wait for all outstanding loads (measured, interleaved runs:
    // 8B gate at B = 2 / 4 / 8 9.99 / 10.83 / 14.70 -> 9.71 / 10.49 / 14.41
    // us, 70B gate at B = 4 35.2 -> 32.3; down and q/o within 1 %).
    auto issue_p = [&](int j) {
        unsigned po, co;
        if constexpr (MULTI) {
            po = co = BUF_OOB;
            if (pf_gb < a.n_gblocks) {
                po = (unsigned)pf_i * pstep + (unsigned)pf_gb * PBLK_B;
                co = (unsigned)pf_i * cstep + (unsigned)pf_gb * CBLK_B;
            }
            if (++pf_i == ntl) {
                pf_i = 0;
                pf_gb += nw;
            }
        } else {
            po = (unsigned)pf_i * pstep + (unsigned)wv * PBLK_B;
            co = (unsigned)pf_i * cstep + (unsigned)wv * CBLK_B;
            ++pf_i;
        }
        P[j] = buf_load16(prs, p_lane + po);
        return co;
    };
    auto issue_c = [&](int j, unsigned co) { C[j] = buf_coef_groups<K>(crs, c_lane + co); };
    auto issue = [&](int j) { issue_c(j, issue_p(j)); };
    // The lane's eight activations of gblock gb for every vector.  One gblock
    // per wavefront: vectors >= B load the last vector again (their limbs are
    // staged but no operand reads them), and lanes past I (ragged end) read a
    // valid address and are zeroed -- only in a gblock that is not full, a
    // wavefront-uniform test -- so the loads need no branches (measured: q/o
    // at B = 2 / 4 / 8 5.0 -> 4.7, 5.9 -> 5.6, 8.1 -> 7.7 us).  Several
    // gblocks per wavefront (the next gblock's load sits in the stream): lanes
    // past I and vectors >= B load nothing and read zero, which measured faster
    // there (8B down at B = 2 11.5 against 12.1 us, 70B down 32.2 against 34.0).
    auto load_x = [&](uint4 *X, int gb) {
        const int e = gb * (GB * GROUP) + lane * 8;
        if constexpr (MULTI) {
            const bool in = e < a.I;
#pragma unroll
            for (int b = 0; b < NB; ++b)
                X[b] = (in && b < B) ? *(const uint4 *)(a.x + (size_t)b * a.I + e) : make_uint4(0u, 0u, 0u, 0u);
        } else {
            const int ec = min(e, a.I - 8);
#pragma unroll
            for (int b = 0; b < NB; ++b)
                X[b] = *(const uint4 *)(a.x + (size_t)min(b, B - 1) * a.I + ec);
            if ((gb + 1) * (GB * GROUP) > a.I) {
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    X[b] = e < a.I ? X[b] : make_uint4(0u, 0u, 0u, 0u);
            }
        }
    };

    uint4 Xc[NB];
    load_x(Xc, wv);
#pragma unroll
    for (int j = 0; j < D; ++j)
        issue(j);
    __builtin_amdgcn_sched_barrier(0);

    *(uint32_t *)(stage + ZERO0 + 4 * lane) = 0u;  // the zero region
    const int ZERO = ZERO0 + 16 * (lane & 15);
    // B operand reads: lane (column n = lane%16 = (vector n/4, limb n%4),
    // k-block lane/16) takes k = 16 kb + [0,16) and 64 + 16 kb + [0,16) of
    // its vector's limb; absent vectors read the zero chunk.
    const int n = lane & 15, kb = lane >> 4;
    const int vb = n >> 2, limb = n & 3;
    // limb writes: lane owns elements 8*lane.. of the gblock = group lane/16,
    // elements 8*(lane%16).. of it
    const int wr_off = (lane >> 4) * (2 * 4 * GROUP) + 8 * (lane & 15);
    const int inv_alpha = inv_alpha_exp(lane & 3);
    // staging phases per column set (vector pairs) and the lane's phase
    constexpr int NPH = (VPS + 1) / 2;
    const int my_phase = min(vb >> 1, NPH - 1);

    v8i Bop[NS][GB];
    float oscale[NS];  // 2^-sigma of the lane's vector, per set
    // With four or more vectors the activation maxima are reduced first, two
    // per register, so that the reductions' latencies overlap, and every
    // vector is split (vectors >= B hold zeros and give zero limbs in their
    // own slots, which no operand reads); with two, each vector present is
    // reduced and split in turn (measured faster there in the kernels that
    // rebuild in the middle of the stream).  The limbs of a vector pair are
    // staged, then the lanes of that pair's columns read their operands.
    auto build = [&](const uint4 *X) {
        uint32_t amax2[(NB + 1) / 2] = {};
        if constexpr (NB >= 4) {
#pragma unroll
            for (int p = 0; p < (NB + 1) / 2; ++p)
                amax2[p] = wave_absmax2_bits(X[2 * p], X[2 * p + 1]);
        }
#pragma unroll
        for (int st = 0; st < NS; ++st) {
            float inv_scale[VPS];
#pragma unroll
            for (int ph = 0; ph < NPH; ++ph) {
#pragma unroll
                for (int vv = 0; vv < 2; ++vv) {
                    const int v = 2 * ph + vv;
                    if (v >= VPS)
                        break;
                    const int b = st * SBS_VPS + v;
                    inv_scale[v] = 1.0f;
                    if (NB >= 4 || b < B) {
                        const float amax = NB >= 4 ? half_bits_to_float((amax2[b / 2] >> (16 * (b & 1))) & 0xffffu)
                                                   : wave_absmax_h(X[b]);
                        const int sigma = scale_exponent(amax);
                        inv_scale[v] = ldexpf(1.0f, -sigma);
                        const Limbs L = split_limbs(X[b], sigma, inv_alpha);
                        unsigned char *dst = stage + wr_off + vv * 4 * GROUP;
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            *(uint2 *)(dst + j * GROUP) = make_uint2(L.l[j][0], L.l[j][1]);
                    }
                }
                // same wavefront: the reads below follow these writes, and the
                // next phase's writes follow the reads
                if (my_phase == ph) {
                    const bool act = vb < VPS && st * SBS_VPS + vb < B;
#pragma unroll
                    for (int g = 0; g < GB; ++g) {
                        const int lo = act ? ((g * 2 + (vb & 1)) * 4 + limb) * GROUP + 16 * kb : ZERO;
                        const int hi = act ? lo + 64 : ZERO;
                        Bop[st][g] = lds_operand(stage + lo, stage + hi);
                    }
                }
            }
            float os = inv_scale[0];
#pragma unroll
            for (int v = 1; v < VPS; ++v)
                os = vb == v ? inv_scale[v] : os;
            oscale[st] = os;
        }
    };
    build(Xc);
    uint4 Xn[MULTI ? NB : 1];
    if constexpr (MULTI)
        load_x(Xn, wv + nw);
    __builtin_amdgcn_sched_barrier(0);

    // red offset of this lane's (row, column) partials: column n = (vector,
    // limb) of its set; the four limbs of a vector are added in the final sum
    float *red_w = red + (wv * NS * TR + (lane >> 4) * NP) * 16 + n;
    const int red_tile = nw * NS * TR * 16;
    int cur_i = 0, cur_gb = wv;
    for (int m0 = 0; m0 < n_items; m0 += D) {
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int m = m0 + j;
            // Items past the end read zero planes and coefficients; only
            // their stores are skipped, so the unrolled body has no branch
            // (apart from the rebuild at a gblock change).
            const bool valid = m < n_items;
            if constexpr (MULTI) {
                if (valid && cur_i == 0 && m > 0) {  // first item of the next gblock
                    build(Xn);
                    load_x(Xn, cur_gb + nw);
                }
            }
            const uint4 pw = transpose_rows4(P[j]);
            const uint32_t words[GB] = {pw.x, pw.y, pw.z, pw.w};
            v4f d[GB][NS];
#pragma unroll
            for (int g = 0; g < GB; ++g) {
                const v8i A = fp4_operand(words[g]);
#pragma unroll
                for (int st = 0; st < NS; ++st)
                    d[g][st] = mfma_fp4_fp8<false>(A, Bop[st][g], v4f{0.f, 0.f, 0.f, 0.f});
            }
            const CoefGroups<K> cr = C[j];
            const unsigned co_next = issue_p(j);
#pragma unroll
            for (int st = 0; st < NS; ++st) {
                // the lane's (tile row, vector, limb) partials of the item:
                // every group's coefficients chained into one accumulator
                float acc[NP];
#pragma unroll
                for (int p = 0; p < NP; ++p)
                    acc[p] = 0.f;
#pragma unroll
                for (int g = 0; g < GB; ++g)
                    fma_coefs<K>(coef_group<K>(cr, g), d[g][st], acc);
                if (valid) {
                    float *r = red_w + cur_i * red_tile + st * TR * 16;
#pragma unroll
                    for (int p = 0; p < NP; ++p) {
                        if (!MULTI || cur_gb == wv)
                            r[p * 16] = acc[p] * oscale[st];
                        else
                            r[p * 16] += acc[p] * oscale[st];
                    }
                }
            }
            issue_c(j, co_next);
            if (valid) {
                if (++cur_i == ntl && MULTI) {
                    cur_i = 0;
                    cur_gb += nw;
                }
            }
        }
    }

    __syncthreads();
    const int row_base = tile0 * TR;
    const int rows = ntl * TR;
    for (int idx = threadIdx.x; idx < rows * B; idx += blockDim.x) {
        const int b = idx / rows, lr = idx % rows;
        const int o = row_base + lr;
        if (o < a.O) {
            const int st = b / SBS_VPS, v = b % SBS_VPS;
            const float *r = red + (lr / TR) * red_tile + (st * TR + lr % TR) * 16 + 4 * v;
            float s = 0.f;
            for (int w = 0; w < nw; ++w) {
                const float4 q = *(const float4 *)(r + w * NS * TR * 16);  // the vector's four limbs
                s += (q.x + q.y) + (q.z + q.w);
            }
            a.y[(size_t)b * a.O + o] = __half_as_ushort(__float2half_rn(s));
        }
    }
}

// Kernels are compiled for NB = 2, 4 and 8 vectors; a call with B vectors
// runs the smallest NB >= B (absent vectors are neither read nor written).
template <int K, int NB, int D>
static const void *sbs_kernel_for(bool multi)
{
    return multi ? (const void *)gemm_sbs_kernel<K, NB, D, true> : (const void *)gemm_sbs_kernel<K, NB, D, false>;
}

template <int K, int D>
static const void *sbs_kernel_kd(int nb, bool multi)
{
    return nb == 2   ? sbs_kernel_for<K, 2, D>(multi)
           : nb == 4 ? sbs_kernel_for<K, 4, D>(multi)
                     : sbs_kernel_for<K, 8, D>(multi);
}

template <int K>
static const void *sbs_kernel_k(int nb, bool multi, bool long_ring)
{
    if (multi && nb <= 4)
        return nb == 2 ? (const void *)gemm_sbs_kernel<K, 2, SBVR_SBS_DEPTH_MULTI_SMALL, true>
                       : (const void *)gemm_sbs_kernel<K, 4, SBVR_SBS_DEPTH_MULTI_SMALL, true>;
    return long_ring ? sbs_kernel_kd<K, SBVR_SBS_DEPTH_LONG>(nb, multi)
                     : sbs_kernel_kd<K, SBVR_SBS_DEPTH_SHORT>(nb, multi);
}

int launch_gemm_sbs(const Dims &d, const void *planes_dev, const void *coeffs_dev,
                    const uint16_t *X, uint16_t *Y, int B, hipStream_t stream)
{
    const int nb = B <= 2 ? 2 : (B <= 4 ? 4 : 8);
    const int gpw = (d.n_gblocks + SBVR_SBS_MAX_WAVES - 1) / SBVR_SBS_MAX_WAVES;
    // several gblocks per wavefront: all eight wavefronts, so that the strided
    // gblock assignment balances the four SIMDs
    const int waves = gpw > 1 ? SBVR_SBS_MAX_WAVES : (d.n_gblocks + gpw - 1) / gpw;
    // tiles per workgroup, capped so that dynamic LDS stays within SBS_LDS_MAX
    const size_t fixed = (size_t)waves * sbs_stage_bytes(nb);
    const size_t per_tile = (size_t)waves * sbs_sets(nb) * d.tr * 16 * 4;
    const int max_tpw = (int)((SBS_LDS_MAX - fixed) / per_tile);
    const int tpw = min((d.n_tiles + SBVR_SBS_GROUPS - 1) / SBVR_SBS_GROUPS, max_tpw);
    const int grid = (d.n_tiles + tpw - 1) / tpw;
    const bool multi = gpw > 1;
    GemvArgs a = {(const uint4 *)planes_dev, (const uint16_t *)coeffs_dev, X, Y, d.O, d.I, d.k,
                  d.n_tiles, d.n_gblocks, gpw, B, tpw};
    const size_t lds = fixed + (size_t)tpw * per_tile;
    const bool long_ring = tpw >= SBVR_SBS_LONG_TPW;
    const void *fn = d.k == 4   ? sbs_kernel_k<4>(nb, multi, long_ring)
                     : d.k == 3 ? sbs_kernel_k<3>(nb, multi, long_ring)
                     : d.k == 2 ? sbs_kernel_k<2>(nb, multi, long_ring)
                                : sbs_kernel_k<1>(nb, multi, long_ring);
    void *args[] = {&a};
    return launch_kernel(fn, dim3(grid), dim3(64 * waves), lds, stream, args);
}

}  // namespace sbvr
