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
// matrix-core instruction), up to 64 tokens (BTT tiles of 16) and a run of
// whole groups of the inner dimension (a K-slice).  A workgroup of 16
// wavefronts holds R = 16 / S row tiles times S K-slices; the S partial sums
// of a row tile are added through LDS at the end in a fixed order
// (deterministic).  Per group a wavefront
//   * builds the 2^k-entry subset-sum table of each of its 16 rows in its own
//     LDS region (binary32 sums, exact when the coefficients span at most 12
//     binades, else binary64; rounded once to binary16);
//   * per 32-element step (word ks of each plane): forms the k-bit subset
//     index of the lane's eight consecutive elements from the plane words (the
//     device bit layout puts element 8v+p of a word at bit 4p+v, so
//     (w >> v) & 0x11111111 holds bit i of elements 8v..8v+7 in nibbles
//     0..7), looks them up, and multiplies the eight binary16 weights with the
//     BTT token tiles of X on v_mfma_f32_16x16x32_f16 (lane l: row or column
//     l % 16, k = 8 (l / 16) .. +7; measured on the device).
// The plane slots, coefficients and activations of the next group are loaded
// while the current one is decoded.
// Bound: for short prompts the weight stream and the decoding (a few vector
// instructions and one LDS lookup per weight and 64-token block); for long
// ones the matrix cores (2 T O I flops) and the activation reads.
#include "device_ops.h"
#include "f16_round.h"
#include "launch.h"

namespace sbvr {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));

// wavefronts per workgroup (R row tiles x S K-slices): 16, or 8 for tiles of
// 32 or 64 tokens, whose double-buffered activations need more registers
__host__ __device__ constexpr int pf_waves(int btt) { return btt >= 2 ? 8 : 16; }

struct PrefillArgs {
    const uint32_t *planes;  // device plane blocks
    const uint16_t *coeffs;  // device coefficient blocks
    const uint16_t *X;       // binary16 [T][I]
    uint16_t *Y;             // binary16 [T][O]
    int O, I, T, n_tiles, n_gblocks, G, gps;  // gps: groups per K-slice
    int S;                                    // K-slices per workgroup (a power of two <= 16)
};

__device__ __forceinline__ int f16_exp(uint32_t h)  // unbiased exponent, subnormals as -14
{
    const int e = (int)((h >> 10) & 0x1f);
    return e == 0 ? -14 : e - 15;
}

template <int K, int BTT>
__global__ void __launch_bounds__(64 * pf_waves(BTT)) prefill_kernel(PrefillArgs a)
{
    constexpr int TR = tile_rows(K), NSUB = 1 << K;
    constexpr int LUT_B = 16 * NSUB * 2;  // per wavefront: [16 rows][subset]
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63, w = wave_id();
    const int S = a.S, R = pf_waves(BTT) / S;
    const int ks_id = w % S, rt = w / S;  // K-slice and row tile of this wavefront
    const int n = lane & 15, kq = lane >> 4;
    uint16_t *lut = (uint16_t *)(smem + w * LUT_B);
    const int o_base = (blockIdx.x * R + rt) * 16, t_base = blockIdx.y * 16 * BTT;
    const int g0 = ks_id * a.gps, g1 = min(a.G, g0 + a.gps);
    const int rows_dev = a.n_tiles * TR;  // rows held by the device format (padding included)

    v4f acc[BTT];
#pragma unroll
    for (int tt = 0; tt < BTT; ++tt)
        acc[tt] = v4f{0.f, 0.f, 0.f, 0.f};

    // the decode row of this lane (its column of the result), and the table
    // entries it builds: row n, subsets NSUB/4 * kq .. (all of them for k < 2)
    const int o = min(o_base + n, rows_dev - 1);
    const bool row_ok = o_base + n < rows_dev;
    const int tile = o / TR, r = o % TR;
    struct GroupLoads {
        uint4 slot[K];
        uint16_t c[K];
        v8h x[4][BTT];  // activations of the four 32-element steps
    };
    // loads of one group, issued a group ahead of their use: the row's plane
    // slots (16 bytes: the group's four words), its coefficients and the
    // token tiles' activations
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
#pragma unroll
        for (int tt = 0; tt < BTT; ++tt) {
            const int t = t_base + 16 * tt + n;
            const uint16_t *xp = a.X + (size_t)min(t, a.T - 1) * a.I + (size_t)g * GROUP + 8 * kq;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                uint4 v = *(const uint4 *)(xp + ks * 32);
                if (t >= a.T)
                    v = make_uint4(0u, 0u, 0u, 0u);
                L.x[ks][tt] = __builtin_bit_cast(v8h, v);
            }
        }
    };

    GroupLoads cur, nxt;
    if (g0 < g1)
        load_group(g0, cur);
    for (int g = g0; g < g1; ++g) {
        if (g + 1 < g1)
            load_group(g + 1, nxt);
        // ---- subset-sum table of the 16 rows for group g ----
        {
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
            constexpr int PER = NSUB >= 4 ? NSUB / 4 : NSUB;  // entries this lane writes
            const int p0 = NSUB >= 4 ? PER * kq : 0;
            uint16_t *lrow = lut + n * NSUB + p0;
            if (emax - emin <= 11) {
                // every subset sum has at most 24 significant bits: exact in
                // binary32, one rounding to binary16
                float cf[K];
#pragma unroll
                for (int i = 0; i < K; ++i)
                    cf[i] = half_bits_to_float(c[i]);
#pragma unroll
                for (int q = 0; q < PER; ++q) {
                    const int p = p0 + q;
                    float sum = 0.f;
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        sum += ((p >> i) & 1) ? cf[i] : 0.f;
                    lrow[q] = __half_as_ushort(__float2half_rn(sum));
                }
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
        }
        // the table is read by other lanes of this wavefront only: its LDS
        // writes complete before the reads below (in order within a wavefront)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        const uint16_t *L = lut + n * NSUB;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            uint32_t pat = 0u;  // nibble p: subset index of element 32 ks + 8 kq + p
#pragma unroll
            for (int i = 0; i < K; ++i) {
                const uint4 sl = cur.slot[i];
                const uint32_t word = ks == 0 ? sl.x : (ks == 1 ? sl.y : (ks == 2 ? sl.z : sl.w));
                pat |= ((word >> kq) & 0x11111111u) << i;
            }
            if (!row_ok)
                pat = 0u;  // rows past the device format: entry 0 (zero)
            uint4 bw;
            bw.x = (uint32_t)L[pat & 0xf] | ((uint32_t)L[(pat >> 4) & 0xf] << 16);
            bw.y = (uint32_t)L[(pat >> 8) & 0xf] | ((uint32_t)L[(pat >> 12) & 0xf] << 16);
            bw.z = (uint32_t)L[(pat >> 16) & 0xf] | ((uint32_t)L[(pat >> 20) & 0xf] << 16);
            bw.w = (uint32_t)L[(pat >> 24) & 0xf] | ((uint32_t)L[pat >> 28] << 16);
            const v8h B = __builtin_bit_cast(v8h, bw);
#pragma unroll
            for (int tt = 0; tt < BTT; ++tt)
                acc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(cur.x[ks][tt], B, acc[tt], 0, 0, 0);
        }
        // the next group's table writes follow this group's lookups (in order)
        if (g + 1 < g1)
            cur = nxt;
    }

    // ---- the S K-slices of each row tile summed in a fixed order: halving
    // tree through LDS (slot of K-slice s of row tile rt: (rt * S/2 + s)) ----
    float *red = (float *)smem;  // [R][S / 2][BTT * 4][64 lanes]
    __syncthreads();
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

template <int K>
static const void *prefill_kernel_for(int btt)
{
    switch (btt) {
    case 1: return (const void *)prefill_kernel<K, 1>;
    case 2: return (const void *)prefill_kernel<K, 2>;
    default: return (const void *)prefill_kernel<K, 4>;
    }
}

// Launch shape: BTT token tiles of 16 per workgroup (1, 2 or 4: prompts of
// more than 64 tokens take several workgroups along the tokens), 16 (8 at
// BTT = 2, 4) wavefronts per workgroup split into R row tiles x S K-slices.  S (a
// power of two, at most the wavefront count and the group count) is the
// largest that keeps the
// grid near 4096 wavefronts (four per SIMD): splitting K further only
// shortens each wavefront's run of groups (its first loads' latency is paid
// per run) and multiplies the activation reads (each row tile reads its
// tokens' activations once).
int launch_prefill(const Dims &d, const void *planes_dev, const void *coeffs_dev, const uint16_t *X, uint16_t *Y,
                   int T, hipStream_t stream)
{
    const int btt = T <= 16 ? 1 : (T <= 32 ? 2 : 4);
    const int gy = (T + 16 * btt - 1) / (16 * btt);
    int S = 1;
    // waves = 16 * ceil(O * S / 256) * gy
    const int waves = pf_waves(btt);
    // total wavefronts = waves * ceil(O * S / (16 * waves)) * gy ~ O * S * gy / 16
    while (2 * S <= waves && 2 * S <= d.G && (long)d.O * 2 * S * gy <= 4096L * 16)
        S *= 2;
    const int R = waves / S;
    const int gx = (d.O + 16 * R - 1) / (16 * R);
    PrefillArgs a = {(const uint32_t *)planes_dev, (const uint16_t *)coeffs_dev, X, Y, d.O, d.I, T, d.n_tiles,
                     d.n_gblocks, d.G, (d.G + S - 1) / S, S};
    const size_t lut = (size_t)waves * 16 * (1u << d.k) * 2;
    const size_t red = (size_t)R * (S / 2) * btt * 4 * 64 * 4;
    const size_t lds = lut > red ? lut : red;
    const void *fn = d.k == 4   ? prefill_kernel_for<4>(btt)
                     : d.k == 3 ? prefill_kernel_for<3>(btt)
                     : d.k == 2 ? prefill_kernel_for<2>(btt)
                                : prefill_kernel_for<1>(btt);
    void *args[] = {&a};
    return launch_kernel(fn, dim3(gx, gy), dim3(64 * waves), lds, stream, args);
}

}  // namespace sbvr
