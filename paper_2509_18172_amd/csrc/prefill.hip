// Prefill GEMM on SBVR weights: Y[t][o] = sum_j X[t][j] * fp16(w_hat[o][j])
// for a prompt of T tokens (the paper's prefill design decompresses the
// weights to binary16 and multiplies them on the tensor cores, Sec. 5.1; here
// the binary16 matrix never goes to memory).
//
// The decoded weight fp16(w_hat) is the correctly rounded subset sum of its
// group's coefficients (Sec. 4.1), the same value sbvr_decompress writes, so
// the result equals X times the decompressed matrix with fp32 accumulation.
//
// Work split.  A wavefront owns 16 weight rows (one column tile of the
// matrix-core instruction), BTT token tiles of 16 (BTT = 1, 2, 4, 8) and a
// run of whole groups of the inner dimension (a K-slice).  A workgroup of 16
// wavefronts holds R = 16 / S row tiles times S K-slices; the S partial sums
// of a row tile are added through LDS at the end in a fixed order.  Per group
//   * the R wavefronts of a K-slice stage the group's activation tile
//     (16 BTT tokens x 128 values) in LDS with coalesced 16-byte loads, double
//     buffered, so the activations are read once per workgroup rather than
//     once per row tile;
//   * a wavefront builds the 2^k-entry subset-sum table of each of its 16 rows
//     in its own LDS region (binary32 sums, exact when the coefficients span at
//     most 12 binades, else binary64; rounded once to binary16);
//   * per 32-element step (word ks of each plane) it forms the k-bit subset
//     index of the lane's eight consecutive elements from the plane words (the
//     device bit layout puts element 8v+p of a word at bit 4p+v, so
//     (w >> v) & 0x11111111 holds bit i of elements 8v..8v+7 in nibbles
//     0..7), looks them up, and multiplies the eight binary16 weights with the
//     BTT token tiles on v_mfma_f32_16x16x32_f16 (lane l: row or column
//     l % 16, k = 8 (l / 16) .. +7; measured on the device).
// The plane slots, coefficients and activations of the next group are loaded
// while the current one is decoded.
// Bound: the decoding (about 300 vector instructions per wavefront and group,
// whatever BTT is); BTT = 8 amortises it over 128 tokens.  From 96 tokens,
// where its grid fills the chip, the long-prompt kernel further down runs
// instead (32 x 32 products, 32-row column tiles).
#include "device_ops.h"
#include "lds_lookup.h"
#include "f16_round.h"
#include "launch.h"

namespace sbvr {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));

constexpr int PF_WAVES = 16;          // wavefronts per workgroup: R row tiles x S K-slices
constexpr int PF_XROW = 256 + 16;     // LDS bytes per token row of an activation tile (padding
                                      // spreads the 16 rows of an operand read over all banks)
// subset-sum table rows padded by two entries (consecutive rows start one
// LDS bank apart; 0, 2 and 4 measured the same)
constexpr int PF_LUT_PAD = 2;
// activation chunks (16 bytes) per thread and group, at most: the launcher
// keeps S BTT <= 4 pf_xpt(BTT) (a K-slice's 1024 / S threads load 256 BTT chunks)
__host__ __device__ constexpr int pf_xpt(int btt) { return btt <= 2 ? 4 : 2; }
constexpr size_t PF_LDS_MAX = 160 * 1024;  // LDS of one workgroup on gfx950

struct PrefillArgs {
    const uint32_t *planes;  // device plane blocks
    const uint16_t *coeffs;  // device coefficient blocks
    const uint16_t *X;       // binary16 [T][I]
    uint16_t *Y;             // binary16 [T][O]
    int O, I, T, n_tiles, n_gblocks, G, gps;  // gps: groups per K-slice
    int S;                                    // K-slices per workgroup (a power of two)
};

// LDS: per K-slice two activation tiles of 16 BTT token rows (PF_XROW bytes
// each: the group's 128 binary16 values), then per wavefront its 16 rows x
// 2^k subset-sum table.  The K-slice reduction reuses the front afterwards.
__host__ __device__ constexpr int pf_xtile(int btt) { return 16 * btt * PF_XROW; }

template <int K, int BTT>
__global__ void __launch_bounds__(64 * PF_WAVES) prefill_kernel(PrefillArgs a)
{
    constexpr int TR = tile_rows(K), NSUB = 1 << K;
    constexpr int LROW = NSUB + PF_LUT_PAD;  // table row stride (binary16 entries)
    constexpr int LUT_B = 16 * LROW * 2;
    constexpr int XT = pf_xtile(BTT);
    constexpr int XCH = 16 * BTT * 16;  // 16-byte chunks of an activation tile
    constexpr int XPT = pf_xpt(BTT);
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63, w = wave_id();
    const int S = a.S, R = PF_WAVES / S;
    const int ks_id = w % S, rt = w / S;  // K-slice and row tile of this wavefront
    const int n = lane & 15, kq = lane >> 4;
    unsigned char *xbuf = smem + (size_t)ks_id * 2 * XT;
    uint16_t *lut = (uint16_t *)(smem + (size_t)S * 2 * XT + w * LUT_B);
    const int o_base = (blockIdx.x * R + rt) * 16, t_base = blockIdx.y * 16 * BTT;
    const int g0 = ks_id * a.gps;
    const int rows_dev = a.n_tiles * TR;  // rows held by the device format (padding included)

    v4f acc[BTT];
#pragma unroll
    for (int tt = 0; tt < BTT; ++tt)
        acc[tt] = v4f{0.f, 0.f, 0.f, 0.f};

    // the decode row of this lane (its column of the result)
    const int o = min(o_base + n, rows_dev - 1);
    const bool row_ok = o_base + n < rows_dev;
    const int tile = o / TR, r = o % TR;
    struct GroupLoads {
        uint4 slot[K];
        uint16_t c[K];
    };
    // the row's plane slots (16 bytes: the group's four words) and coefficients
    auto load_group = [&](int g, GroupLoads &L) {
        const int gb = g / GB, b = g % GB;
        const size_t blk = (size_t)tile * a.n_gblocks + gb;
        const uint4 *sp = (const uint4 *)(a.planes + blk * plane_block_words(K)) + (b * TR + r) * K;
#pragma unroll
        for (int i = 0; i < K; ++i)
            L.slot[i] = sp[i];
        const uint16_t *cp = a.coeffs + blk * coeff_block_entries(K) + coeff_entry(K, r, b, 0);  // contiguous
#pragma unroll
        for (int i = 0; i < K; ++i)
            L.c[i] = cp[i];
    };
    // a group's activation tile, loaded by the K-slice's R wavefronts: 16
    // consecutive threads read one token's 256 bytes (tokens past T read as
    // zero)
    const int xthr = rt * 64 + lane, nxthr = R * 64;
    // (no per-lane branch: chunks past the tile or the prompt read the last
    // token and are zeroed; rounds past the chunks of the tile's tokens, the
    // same for every thread of the workgroup, are skipped)
    const int x_rounds = (min(XCH, (a.T - t_base) * 16) + nxthr - 1) / nxthr;
    auto load_x = [&](int g, uint4 *v) {
#pragma unroll
        for (int q = 0; q < XPT; ++q) {
            v[q] = make_uint4(0u, 0u, 0u, 0u);
            if (q < x_rounds) {
                const int ch = xthr + q * nxthr;
                const int t = t_base + ch / 16;
                const uint4 r =
                    *(const uint4 *)(a.X + (size_t)min(t, a.T - 1) * a.I + (size_t)g * GROUP + (ch % 16) * 8);
                v[q] = ch < XCH && t < a.T ? r : make_uint4(0u, 0u, 0u, 0u);
            }
        }
    };
    auto store_x = [&](unsigned char *buf, const uint4 *v) {
#pragma unroll
        for (int q = 0; q < XPT; ++q) {
            const int ch = xthr + q * nxthr;
            if (ch < XCH)
                *(uint4 *)(buf + (ch / 16) * PF_XROW + (ch % 16) * 16) = v[q];
        }
    };

    // every wavefront of the workgroup runs gps steps (groups past G are
    // skipped but keep the barriers aligned)
    // Every load is issued unconditionally (past the K-slice's last group the
    // current or last group is loaded again and not used): with no branch
    // around them the compiler's load counters stay exact through the loop,
    // so the next group's loads overlap this group's products instead of
    // being waited for before its table build.
    GroupLoads cur, nxt;
    uint4 xv[XPT];
    const int g_first = min(g0, a.G - 1);
    load_group(g_first, cur);
    load_x(g_first, xv);
    store_x(xbuf, xv);
    __syncthreads();
    for (int j = 0; j < a.gps; ++j) {
        const int g = g0 + j;
        const bool more = j + 1 < a.gps && g + 1 < a.G;
        const int gn = more ? g + 1 : min(g, a.G - 1);
        load_group(gn, nxt);
        load_x(gn, xv);  // stored after this group's products
        if (g < a.G) {
            // ---- subset-sum table of the 16 rows for group g (lane: row n,
            // subsets NSUB/4 * kq ..; all of them for k < 2) ----
            uint32_t c[K];
#pragma unroll
            for (int i = 0; i < K; ++i)
                c[i] = row_ok ? (uint32_t)cur.c[i] : 0u;
            int emax = -30, emin = 30;
#pragma unroll
            for (int i = 0; i < K; ++i) {
                if (c[i] & 0x7fffu) {
                    emax = max(emax, f16_exp(c[i]));
                    emin = min(emin, f16_exp(c[i]));
                }
            }
            constexpr int PER = NSUB >= 4 ? NSUB / 4 : NSUB;
            const int p0 = NSUB >= 4 ? PER * kq : 0;
            uint16_t *lrow = lut + n * LROW + p0;
            // binary32 path: every subset sum has at most 24 significant bits
            // (exact whatever the order of the additions), one rounding to
            // binary16.  The entry index is p0 + q: its bits above LOGPER come
            // from the lane (p0), the ones below from q (compile time).
            constexpr int LOGPER = PER == 4 ? 2 : (PER == 2 ? 1 : 0);
            auto table32 = [&]() {
                float cf[K];
#pragma unroll
                for (int i = 0; i < K; ++i)
                    cf[i] = half_bits_to_float(c[i]);
                float hi = 0.f;
#pragma unroll
                for (int i = LOGPER; i < K; ++i)
                    hi += ((p0 >> i) & 1) ? cf[i] : 0.f;
#pragma unroll
                for (int q = 0; q < PER; ++q) {
                    float sum = hi;
#pragma unroll
                    for (int i = 0; i < LOGPER && i < K; ++i)
                        if ((q >> i) & 1)
                            sum += cf[i];
                    lrow[q] = __half_as_ushort(__float2half_rn(sum));
                }
            };
            const bool wide = emax - emin > 11;
            if (__builtin_amdgcn_ballot_w64(wide) == 0) {
                table32();  // no lane of the wavefront needs binary64 (wavefront-uniform branch)
            } else if (!wide) {
                table32();
            } else {
#pragma unroll
                for (int q = 0; q < PER; ++q) {
                    const int p = p0 + q;
                    double sum = 0.0;  // exact: at most K binary16 terms
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        sum += ((p >> i) & 1) ? (double)half_bits_to_float(c[i]) : 0.0;
                    lrow[q] = f64_to_f16_rne(sum);
                }
            }
            // the table is read by other lanes of this wavefront only: its LDS
            // writes complete before the reads below (in order within a wavefront)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

            const uint16_t *L = lut + n * LROW;
            const unsigned char *xt = xbuf + (j & 1) * XT;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                uint32_t pat = 0u;  // nibble p: subset index of element 32 ks + 8 kq + p
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    const uint4 sl = cur.slot[i];
                    const uint32_t word = ks == 0 ? sl.x : (ks == 1 ? sl.y : (ks == 2 ? sl.z : sl.w));
                    pat |= ((word >> kq) & 0x11111111u) << i;
                }
                // (rows past the device format have all-zero tables.)  Byte b
                // of e2 / o2 is the byte offset of nibble 2b / 2b+1's entry,
                // so each lookup's address is one byte-select add; the entries
                // load straight into the halves of the operand registers.
                const uint32_t e2 = (pat & 0x0F0F0F0Fu) << 1, o2 = (pat >> 3) & 0x1E1E1E1Eu;
                const uint32_t Lbase = lds_addr(L);  // the row's table
                const uint32_t a[8] = {add_byte<0>(Lbase, e2), add_byte<0>(Lbase, o2), add_byte<1>(Lbase, e2),
                                       add_byte<1>(Lbase, o2), add_byte<2>(Lbase, e2), add_byte<2>(Lbase, o2),
                                       add_byte<3>(Lbase, e2), add_byte<3>(Lbase, o2)};
                auto at = [&](int i) { return *(const __attribute__((address_space(3))) _Float16 *)(uintptr_t)a[i]; };
                const v8h B = {at(0), at(1), at(2), at(3), at(4), at(5), at(6), at(7)};
#pragma unroll
                for (int tt = 0; tt < BTT; ++tt) {
                    // token 16 tt + n, elements 32 ks + 8 kq .. +7
                    const uint4 av = *(const uint4 *)(xt + (16 * tt + n) * PF_XROW + (ks * 4 + kq) * 16);
                    acc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(v8h, av), B, acc[tt], 0,
                                                                      0, 0);
                }
            }
        }
        // the other buffer was last read before the previous barrier
        store_x(xbuf + ((j + 1) & 1) * XT, xv);
        cur = nxt;
        __syncthreads();
    }

    // ---- the S K-slices of each row tile summed in a fixed order: halving
    // tree through LDS (slot of K-slice s of row tile rt: rt * S/2 + s) ----
    float *red = (float *)smem;  // [R][S / 2][BTT * 4][64 lanes]
    for (int half = S / 2; half >= 1; half /= 2) {
        if (ks_id >= half && ks_id < 2 * half) {
            float *dst = red + ((size_t)rt * (S / 2) + (ks_id - half)) * (BTT * 4 * 64);
#pragma unroll
            for (int tt = 0; tt < BTT; ++tt)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    dst[(tt * 4 + e) * 64 + lane] = acc[tt][e];
        }
        __syncthreads();
        if (ks_id < half) {
            const float *src = red + ((size_t)rt * (S / 2) + ks_id) * (BTT * 4 * 64);
#pragma unroll
            for (int tt = 0; tt < BTT; ++tt)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[tt][e] += src[(tt * 4 + e) * 64 + lane];
        }
        __syncthreads();
    }
    if (ks_id != 0)
        return;
    // lane (column n, k-block kq) holds rows (tokens) 4 kq .. 4 kq + 3 of each tile
    const int oo = o_base + n;
#pragma unroll
    for (int tt = 0; tt < BTT; ++tt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t = t_base + 16 * tt + 4 * kq + e;
            if (oo < a.O && t < a.T)
                a.Y[(size_t)t * a.O + oo] = __half_as_ushort(__float2half_rn(acc[tt][e]));
        }
}

// ---------------------------------------------------------------------------
// Long prompts: v_mfma_f32_32x32x16_f16.  The kernel above reads a 16-token
// activation operand from LDS for every 16 x 16 product, and each wavefront
// decodes its weights for at most 128 tokens; past about a hundred tokens the
// LDS reads and the decoding bound it.  Here a wavefront owns RT column tiles
// of 32 weight rows and TT token tiles of 32: each activation operand read
// meets 32 RT rows and each decoded weight 32 TT tokens.  A workgroup of
// PL_WAVES wavefronts holds R = PL_WAVES / S row groups times S K-slices
// (their partial sums added through LDS in a fixed order, as above).  Per
// group a wavefront builds the subset-sum tables of its 32 RT rows (lane: row
// lane % 32, half of the subsets), then per 16-element step each lane looks
// up the eight elements 8 (lane / 32) .. +7 of each of its rows (the device
// bit layout holds them as bits v, v + 4, .., v + 28 of one plane word, v =
// 2 (step % 2) + lane / 32) and issues RT x TT instructions (operand A: 32
// tokens x 16 values, lane: token lane % 32, values 8 (lane / 32) ..; operand
// B: the decoded weights, lane: row lane % 32, the same values).  Result
// register j of a lane holds token 8 (j / 4) + 4 (lane / 32) + j % 4 of the
// tile, row lane % 32.
// ---------------------------------------------------------------------------
constexpr int PL_WAVES = 8;
// activation chunks (16 bytes) per thread and group: S TT (a K-slice's
// 512 / S threads load 512 TT chunks).  The launcher keeps S TT <= 8 for one
// column tile of 64 or 128 tokens (so that its products can split K four and
// two ways) and <= 4 otherwise; a kernel instance holds 4 or 8 chunks (XPT),
// 4 whenever S TT allows (the 8-chunk build of the same shape measured 3-5 %
// slower; 2 x 2 tiles with 8 chunks and four K-slices, 5-10 % slower than
// 1 x 2 tiles with two)
__host__ __device__ constexpr int pl_xpt(int tt) { return tt == 1 ? 4 : 8; }
// instructions per step and wavefront (RT TT) at most: the RT TT x 16
// accumulators of 2 x 2 and 1 x 4 fit the 256 registers of a wavefront at two
// per SIMD; 2 x 4 would spill
constexpr int PL_TILE_MAX = 4;

typedef float v16f __attribute__((ext_vector_type(16)));

__host__ __device__ constexpr int pl_xtile(int tt) { return 32 * tt * PF_XROW; }

template <int K, int RT, int TT, int XPT>
__global__ void __launch_bounds__(64 * PL_WAVES) prefill_long_kernel(PrefillArgs a)
{
    constexpr int TR = tile_rows(K), NSUB = 1 << K;
    constexpr int LROW = NSUB + PF_LUT_PAD;
    constexpr int LUT_B = 32 * RT * LROW * 2;  // a wavefront's tables
    constexpr int XT = pl_xtile(TT);
    constexpr int XCH = 32 * TT * 16;
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63, w = wave_id();
    const int S = a.S, R = PL_WAVES / S;
    const int ks_id = w % S, rg = w / S;  // K-slice and row group of this wavefront
    const int n = lane & 31, kh = lane >> 5;
    unsigned char *xbuf = smem + (size_t)ks_id * 2 * XT;
    uint16_t *lut = (uint16_t *)(smem + (size_t)S * 2 * XT + w * LUT_B);
    const int o_base = (blockIdx.x * R + rg) * 32 * RT, t_base = blockIdx.y * 32 * TT;
    const int g0 = ks_id * a.gps;
    const int rows_dev = a.n_tiles * TR;

    v16f acc[RT][TT];
#pragma unroll
    for (int q = 0; q < RT; ++q)
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[q][tt][e] = 0.f;

    // the lane's decode rows (row lane % 32 of each column tile)
    int tile[RT], rr[RT];
    bool row_ok[RT];
#pragma unroll
    for (int q = 0; q < RT; ++q) {
        const int o = min(o_base + 32 * q + n, rows_dev - 1);
        row_ok[q] = o_base + 32 * q + n < rows_dev;
        tile[q] = o / TR;
        rr[q] = o % TR;
    }
    struct GroupLoads {
        uint4 slot[RT][K];
        uint16_t c[RT][K];
    };
    auto load_group = [&](int g, GroupLoads &L) {
        const int gb = g / GB, b = g % GB;
#pragma unroll
        for (int q = 0; q < RT; ++q) {
            const size_t blk = (size_t)tile[q] * a.n_gblocks + gb;
            const uint4 *sp = (const uint4 *)(a.planes + blk * plane_block_words(K)) + (b * TR + rr[q]) * K;
#pragma unroll
            for (int i = 0; i < K; ++i)
                L.slot[q][i] = sp[i];
            const uint16_t *cp = a.coeffs + blk * coeff_block_entries(K) + coeff_entry(K, rr[q], b, 0);
#pragma unroll
            for (int i = 0; i < K; ++i)
                L.c[q][i] = cp[i];
        }
    };
    // a group's activation tile, loaded by the K-slice's R wavefronts: 16
    // consecutive threads read one token's 256 bytes (tokens past T read zero)
    const int xthr = rg * 64 + lane, nxthr = R * 64;
    // (no per-lane branch: chunks past the tile or the prompt read the last
    // token and are zeroed; rounds past the chunks of the tile's tokens, the
    // same for every thread of the workgroup, are skipped)
    const int x_rounds = (min(XCH, (a.T - t_base) * 16) + nxthr - 1) / nxthr;
    auto load_x = [&](int g, uint4 *v) {
#pragma unroll
        for (int q = 0; q < XPT; ++q) {
            v[q] = make_uint4(0u, 0u, 0u, 0u);
            if (q < x_rounds) {
                const int ch = xthr + q * nxthr;
                const int t = t_base + ch / 16;
                const uint4 r =
                    *(const uint4 *)(a.X + (size_t)min(t, a.T - 1) * a.I + (size_t)g * GROUP + (ch % 16) * 8);
                v[q] = ch < XCH && t < a.T ? r : make_uint4(0u, 0u, 0u, 0u);
            }
        }
    };
    auto store_x = [&](unsigned char *buf, const uint4 *v) {
#pragma unroll
        for (int q = 0; q < XPT; ++q) {
            const int ch = xthr + q * nxthr;
            if (ch < XCH)
                *(uint4 *)(buf + (ch / 16) * PF_XROW + (ch % 16) * 16) = v[q];
        }
    };

    // Every load is issued unconditionally (past the K-slice's last group the
    // current or last group is loaded again and not used): with no branch
    // around them the compiler's load counters stay exact through the loop,
    // so the next group's loads overlap this group's products instead of
    // being waited for before its table build.
    GroupLoads cur, nxt;
    uint4 xv[XPT];
    const int g_first = min(g0, a.G - 1);
    load_group(g_first, cur);
    load_x(g_first, xv);
    store_x(xbuf, xv);
    __syncthreads();
    for (int j = 0; j < a.gps; ++j) {
        const int g = g0 + j;
        const bool more = j + 1 < a.gps && g + 1 < a.G;
        const int gn = more ? g + 1 : min(g, a.G - 1);
        load_group(gn, nxt);
        load_x(gn, xv);  // stored after this group's products
        if (g < a.G) {
            // ---- subset-sum tables of the wavefront's rows for group g (lane:
            // row lane % 32 of each column tile, subsets PER * (lane / 32) ..) ----
            constexpr int PER = NSUB / 2, LOGPER = K - 1;
            const int p0 = PER * kh;
#pragma unroll
            for (int q = 0; q < RT; ++q) {
                uint32_t c[K];
#pragma unroll
                for (int i = 0; i < K; ++i)
                    c[i] = row_ok[q] ? (uint32_t)cur.c[q][i] : 0u;
                int emax = -30, emin = 30;
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    if (c[i] & 0x7fffu) {
                        emax = max(emax, f16_exp(c[i]));
                        emin = min(emin, f16_exp(c[i]));
                    }
                }
                uint16_t *lrow = lut + (32 * q + n) * LROW + p0;
                // binary32 sums (exact when the coefficients span at most 12
                // binades: every subset sum then has at most 24 significant
                // bits), one rounding to binary16; entry p0 + e takes its top
                // bit from the lane and the others from e
                auto table32 = [&]() {
                    float cf[K];
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        cf[i] = half_bits_to_float(c[i]);
                    const float hi = kh ? cf[K - 1] : 0.f;
#pragma unroll
                    for (int e = 0; e < PER; ++e) {
                        float sum = hi;
#pragma unroll
                        for (int i = 0; i < LOGPER; ++i)
                            if ((e >> i) & 1)
                                sum += cf[i];
                        lrow[e] = __half_as_ushort(__float2half_rn(sum));
                    }
                };
                const bool wide = emax - emin > 11;
                if (__builtin_amdgcn_ballot_w64(wide) == 0) {
                    table32();  // no lane needs binary64 (wavefront-uniform branch)
                } else if (!wide) {
                    table32();
                } else {
#pragma unroll
                    for (int e = 0; e < PER; ++e) {
                        const int p = p0 + e;
                        double sum = 0.0;  // exact: at most K binary16 terms
#pragma unroll
                        for (int i = 0; i < K; ++i)
                            sum += ((p >> i) & 1) ? (double)half_bits_to_float(c[i]) : 0.0;
                        lrow[e] = f64_to_f16_rne(sum);
                    }
                }
            }
            // the tables are read by other lanes of this wavefront only: its
            // LDS writes complete before the reads below (in order within a
            // wavefront)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

            const unsigned char *xt = xbuf + (j & 1) * XT;
            // Operands of step st: the lane's eight weights of each of its
            // rows (table lookups) and its activation fragment of each token
            // tile.  Software-pipelined: step st + 1's LDS reads are issued
            // before step st's products, so their latency overlaps the
            // matrix-core work instead of stalling every instruction.
            v8h Bw[2][RT];
            uint4 Av[2][TT];
            auto load_step = [&](int st, v8h *bw, uint4 *av) {
                const int v = 2 * (st & 1) + kh;
#pragma unroll
                for (int q = 0; q < RT; ++q) {
                    uint32_t pat = 0u;  // nibble p: subset index of element 16 st + 8 kh + p
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const uint4 sl = cur.slot[q][i];
                        const int wi = st >> 1;
                        const uint32_t word = wi == 0 ? sl.x : (wi == 1 ? sl.y : (wi == 2 ? sl.z : sl.w));
                        pat |= ((word >> v) & 0x11111111u) << i;
                    }
                    // byte b of e2 / o2: byte offset of nibble 2b / 2b+1's entry
                    const uint32_t e2 = (pat & 0x0F0F0F0Fu) << 1, o2 = (pat >> 3) & 0x1E1E1E1Eu;
                    const uint32_t Lbase = lds_addr(lut + (32 * q + n) * LROW);
                    const uint32_t ad[8] = {add_byte<0>(Lbase, e2), add_byte<0>(Lbase, o2), add_byte<1>(Lbase, e2),
                                            add_byte<1>(Lbase, o2), add_byte<2>(Lbase, e2), add_byte<2>(Lbase, o2),
                                            add_byte<3>(Lbase, e2), add_byte<3>(Lbase, o2)};
                    auto at = [&](int i) {
                        return *(const __attribute__((address_space(3))) _Float16 *)(uintptr_t)ad[i];
                    };
                    bw[q] = v8h{at(0), at(1), at(2), at(3), at(4), at(5), at(6), at(7)};
                }
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)  // token 32 tt + n, elements 16 st + 8 kh .. +7
                    av[tt] = *(const uint4 *)(xt + (32 * tt + n) * PF_XROW + (2 * st + kh) * 16);
            };
            load_step(0, Bw[0], Av[0]);
#pragma unroll
            for (int st = 0; st < 8; ++st) {
                if (st + 1 < 8)
                    load_step(st + 1, Bw[(st + 1) & 1], Av[(st + 1) & 1]);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                    for (int q = 0; q < RT; ++q)
                        acc[q][tt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(v8h, Av[st & 1][tt]),
                                                                            Bw[st & 1][q], acc[q][tt], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // the other buffer was last read before the previous barrier
        store_x(xbuf + ((j + 1) & 1) * XT, xv);
        cur = nxt;
        __syncthreads();
    }

    // ---- the S K-slices of each row group summed in a fixed order (halving
    // tree through LDS; slot of K-slice s of row group rg: rg * S/2 + s) ----
    constexpr int NV = RT * TT * 16;  // values per lane
    float *red = (float *)smem;       // [R][S / 2][NV][64 lanes]
    for (int half = S / 2; half >= 1; half /= 2) {
        if (ks_id >= half && ks_id < 2 * half) {
            float *dst = red + ((size_t)rg * (S / 2) + (ks_id - half)) * (NV * 64);
#pragma unroll
            for (int q = 0; q < RT; ++q)
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        dst[((q * TT + tt) * 16 + e) * 64 + lane] = acc[q][tt][e];
        }
        __syncthreads();
        if (ks_id < half) {
            const float *src = red + ((size_t)rg * (S / 2) + ks_id) * (NV * 64);
#pragma unroll
            for (int q = 0; q < RT; ++q)
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        acc[q][tt][e] += src[((q * TT + tt) * 16 + e) * 64 + lane];
        }
        __syncthreads();
    }
    if (ks_id != 0)
        return;
#pragma unroll
    for (int q = 0; q < RT; ++q) {
        const int oo = o_base + 32 * q + n;
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int t = t_base + 32 * tt + 8 * (e / 4) + 4 * kh + e % 4;
                if (oo < a.O && t < a.T)
                    a.Y[(size_t)t * a.O + oo] = __half_as_ushort(__float2half_rn(acc[q][tt][e]));
            }
    }
}

template <int K>
static const void *prefill_long_kernel_for(int rt, int tt, int S)
{
    const bool wide = S * tt > 4;
    if (rt == 2)
        return tt == 2 ? (const void *)prefill_long_kernel<K, 2, 2, 4> : (const void *)prefill_long_kernel<K, 2, 1, 4>;
    if (tt == 4)
        return wide ? (const void *)prefill_long_kernel<K, 1, 4, 8> : (const void *)prefill_long_kernel<K, 1, 4, 4>;
    if (tt == 2)
        return wide ? (const void *)prefill_long_kernel<K, 1, 2, 8> : (const void *)prefill_long_kernel<K, 1, 2, 4>;
    return (const void *)prefill_long_kernel<K, 1, 1, 4>;
}

template <int K>
static const void *prefill_kernel_for(int btt)
{
    switch (btt) {
    case 1: return (const void *)prefill_kernel<K, 1>;
    case 2: return (const void *)prefill_kernel<K, 2>;
    case 4: return (const void *)prefill_kernel<K, 4>;
    default: return (const void *)prefill_kernel<K, 8>;
    }
}

// Launch shape.  A wavefront's per-group work (plane loads, table build,
// pattern extraction and lookups) is the same whatever BTT is, so large token
// tiles amortise it; splitting K into S slices spreads it over more
// wavefronts and shortens each one's chain of groups; both are bounded by the
// activation tiles' LDS (S BTT <= 4 pf_xpt).  Workgroups hold 1024 threads and
// up to 148 KiB of LDS, one per CU: among the shapes whose grid fits one
// round of the 256 CUs the one with the most workgroups wins (ties: the
// largest S BTT); when none fits, the fewest workgroups.  This rule picks the
// measured best of every (BTT, S) on the Llama-3-8B projection shapes at
// 1 .. 512 tokens.
constexpr int PF_CUS = 256;

// Prompts of at least this many tokens run the long-prompt kernel.
#ifndef SBVR_PF_LONG_MIN_T
#define SBVR_PF_LONG_MIN_T 96
#endif
// ... and its grid has at least this many workgroups (else the kernel above)
#ifndef SBVR_PF_LONG_MIN_WG
#define SBVR_PF_LONG_MIN_WG 192
#endif
// Sweeps: a fixed long-kernel shape (column tiles, token tiles, K-slices);
// 0 lets the rule below choose.
#ifndef SBVR_PF_LONG_RT
#define SBVR_PF_LONG_RT 0
#endif
#ifndef SBVR_PF_LONG_TT
#define SBVR_PF_LONG_TT 0
#endif
#ifndef SBVR_PF_LONG_S
#define SBVR_PF_LONG_S 0
#endif

static size_t prefill_long_lds(int k, int rt, int tt, int S)
{
    const size_t front = (size_t)S * 2 * pl_xtile(tt);
    const size_t red = (size_t)(PL_WAVES / S) * (S / 2) * rt * tt * 16 * 64 * 4;
    return (front > red ? front : red) + (size_t)PL_WAVES * 32 * rt * ((1u << k) + PF_LUT_PAD) * 2;
}

// Long-prompt launch shape: among the (RT, TT, S) whose LDS fits, the grids
// that fit one round of the 256 CUs win, and among those the most workgroups,
// then the widest token tile (each weight is decoded once per token tile),
// then 4 activation chunks per thread over 8, then the largest tile per
// wavefront (RT TT); when none fits, the fewest
// workgroups.  Returns the workgroup count (0: no shape fits).
struct LongShape {
    int rt, tt, S, wg;
};

static LongShape prefill_long_shape(const Dims &d, int T)
{
    LongShape b = {0, 0, 0, 0};
    for (int r = 1; r <= 2; ++r)
        for (int t = 1; t <= 4; t *= 2)
            for (int sk = 1; sk <= PL_WAVES && sk <= d.G && sk * t <= pl_xpt(t); sk *= 2) {
                if (r * t > PL_TILE_MAX)
                    continue;
                if (r == 2 && sk * t > 4)  // two column tiles: 4 chunks per thread only
                    continue;
                if (SBVR_PF_LONG_RT && r != SBVR_PF_LONG_RT)
                    continue;
                if (SBVR_PF_LONG_TT && t != SBVR_PF_LONG_TT)
                    continue;
                if (SBVR_PF_LONG_S && sk != SBVR_PF_LONG_S)
                    continue;
                if (prefill_long_lds(d.k, r, t, sk) > PF_LDS_MAX)
                    continue;
                const int rows = 32 * r * (PL_WAVES / sk);
                const int wg = (d.O + rows - 1) / rows * ((T + 32 * t - 1) / (32 * t));
                const bool fits = wg <= PF_CUS, best_fits = b.wg > 0 && b.wg <= PF_CUS;
                bool take;
                if (b.rt == 0)
                    take = true;
                else if (fits != best_fits)
                    take = fits;
                else if (wg != b.wg)
                    take = fits ? wg > b.wg : wg < b.wg;
                else if (t != b.tt)
                    take = t > b.tt;
                else if ((sk * t <= 4) != (b.S * b.tt <= 4))
                    take = sk * t <= 4;
                else
                    take = r * t > b.rt * b.tt;
                if (take)
                    b = {r, t, sk, wg};
            }
    return b;
}

static int launch_prefill_long(const Dims &d, const LongShape &sh, const void *planes_dev, const void *coeffs_dev,
                               const uint16_t *X, uint16_t *Y, int T, hipStream_t stream)
{
    const int rows = 32 * sh.rt * (PL_WAVES / sh.S);
    const int gx = (d.O + rows - 1) / rows, gy = (T + 32 * sh.tt - 1) / (32 * sh.tt);
    PrefillArgs a = {(const uint32_t *)planes_dev, (const uint16_t *)coeffs_dev, X, Y, d.O, d.I, T, d.n_tiles,
                     d.n_gblocks, d.G, (d.G + sh.S - 1) / sh.S, sh.S};
    const void *fn = d.k == 4   ? prefill_long_kernel_for<4>(sh.rt, sh.tt, sh.S)
                     : d.k == 3 ? prefill_long_kernel_for<3>(sh.rt, sh.tt, sh.S)
                     : d.k == 2 ? prefill_long_kernel_for<2>(sh.rt, sh.tt, sh.S)
                                : prefill_long_kernel_for<1>(sh.rt, sh.tt, sh.S);
    void *args[] = {&a};
    return launch_kernel(fn, dim3(gx, gy), dim3(64 * PL_WAVES), prefill_long_lds(d.k, sh.rt, sh.tt, sh.S), stream,
                         args);
}

int launch_prefill(const Dims &d, const void *planes_dev, const void *coeffs_dev, const uint16_t *X, uint16_t *Y,
                   int T, hipStream_t stream)
{
    // the long-prompt kernel where its grid fills most of the chip (measured:
    // faster there -- Llama-3-8B gate at 128 / 256 / 512 tokens 66.6 / 122 /
    // 167 us -> 60.6 / 94 / 132, down at 512 216 -> 187, q/o 66 -> 57 --,
    // slower for a 1024-row matrix at 128 tokens, whose best long grid has 64
    // workgroups: 16.2 -> 27.5 us)
    if (T >= SBVR_PF_LONG_MIN_T) {
        const LongShape sh = prefill_long_shape(d, T);
        if (sh.wg >= SBVR_PF_LONG_MIN_WG)
            return launch_prefill_long(d, sh, planes_dev, coeffs_dev, X, Y, T, stream);
    }
    int btt = 0, S = 0, best_wg = 0;
    for (int bt = 1; bt <= 8; bt *= 2) {
        if (bt > 1 && 16 * (bt / 2) >= T)  // a smaller tile already covers the prompt
            break;
        const int gy = (T + 16 * bt - 1) / (16 * bt);
        for (int sk = 1; sk <= PF_WAVES && sk <= d.G && sk * bt <= 4 * pf_xpt(bt); sk *= 2) {
            const int wg = (d.O + 16 * (PF_WAVES / sk) - 1) / (16 * (PF_WAVES / sk)) * gy;
            const bool fits = wg <= PF_CUS, best_fits = best_wg > 0 && best_wg <= PF_CUS;
            bool take;
            if (btt == 0)
                take = true;
            else if (fits != best_fits)
                take = fits;
            else if (wg != best_wg)
                take = fits ? wg > best_wg : wg < best_wg;
            else
                take = sk * bt > S * btt;
            if (take) {
                btt = bt;
                S = sk;
                best_wg = wg;
            }
        }
    }
    const int R = PF_WAVES / S;
    const int gx = (d.O + 16 * R - 1) / (16 * R), gy = (T + 16 * btt - 1) / (16 * btt);
    PrefillArgs a = {(const uint32_t *)planes_dev, (const uint16_t *)coeffs_dev, X, Y, d.O, d.I, T, d.n_tiles,
                     d.n_gblocks, d.G, (d.G + S - 1) / S, S};
    const size_t front = (size_t)S * 2 * pf_xtile(btt);
    const size_t red = (size_t)R * (S / 2) * btt * 4 * 64 * 4;
    const size_t lds = (front > red ? front : red) + (size_t)PF_WAVES * 16 * ((1u << d.k) + PF_LUT_PAD) * 2;
    if (lds > PF_LDS_MAX)
        return SBVR_E_UNSUPPORTED;
    const void *fn = d.k == 4   ? prefill_kernel_for<4>(btt)
                     : d.k == 3 ? prefill_kernel_for<3>(btt)
                     : d.k == 2 ? prefill_kernel_for<2>(btt)
                                : prefill_kernel_for<1>(btt);
    void *args[] = {&a};
    return launch_kernel(fn, dim3(gx, gy), dim3(64 * PF_WAVES), lds, stream, args);
}

}  // namespace sbvr
