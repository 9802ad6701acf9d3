// SBVR encoding (Algorithm 1 with the bitvector assignment of Sec. 4.2) on
// the GPU: for every 128-weight group, search the coefficient sets of the
// (r, s, b) grid (Eqs. 4-11) for the one with the smallest mean squared error
// of nearest-subset-sum reconstruction, then give each weight the pattern of
// its nearest subset sum.
//
// The arithmetic is the search's definition carried out in binary64 in a
// fixed order, so the result is bit-identical to any implementation that
// follows the same definition (this file is compiled without floating-point
// contraction):
//   - group statistics in element order: min, max, sum; mean = sum / n;
//   - q95: the linearly interpolated 95th percentile of the sorted group,
//     s[lo] + frac * (s[lo+1] - s[lo]) at position 0.95 (n - 1);
//   - S_j = s_min + (j+1) s_gran, s_min = 2 q95, s_max = 1.1 (max - min),
//     s_gran = (s_max - s_min) / N_scale (Eqs. 6, 8, 10, 11);
//     B_k = b_min + k b_gran, b_max = 2 |mean| / K, b_min = -b_max,
//     b_gran = (b_max - b_min) / N_bias (Eqs. 7, 9, 10, 11);
//     R: -1 + (i+1) (0.5 / N_1) for i < N_1, then -2 + i (1 / N_2) for i < N_2;
//   - entry coefficients c_i = fp16((s r^i) / N(r) + b), r^i by repeated
//     multiplication, N(r) = sum_i abs(r^i) accumulated in i order (1 for the
//     literal form of Eq. 4); entries with s <= 0 or a non-finite c are skipped;
//   - subset sums in bit order, nearest = first strict minimum of
//     abs(x - sum_p) over p ascending, MSE = (sum_j (x_j - sum)^2 in j order) / n,
//     best entry = first strict minimum over entries in (r, s, b) order;
//   - no admissible entry: c = (fp16(mean), 0, ...).
//
// The search needs only each element's smallest squared distance to a subset
// sum, min_p fl((x - sum_p)^2), which equals the square of the nearest
// difference (the rounded square is monotone in |d|); the pattern itself is
// found once, for the chosen entry.
//
// Work split: one wavefront per group; lane l evaluates entries l, l+64, ...
// (each entry's error sum runs over the elements in order, so entries -- not
// elements -- are what is parallel), then the wavefront picks the smallest
// error with the lowest entry index, which is the sequential first minimum.
// The group's values sit in LDS and are read as broadcasts.
#include "device_ops.h"
#include "f16_round.h"
#include "launch.h"

#include <climits>

namespace sbvr {

constexpr int ENC_THREADS = 64;  // one wavefront per group

__device__ __forceinline__ double f16_bits_to_double(uint16_t h)
{
    return (double)half_bits_to_float(h);  // both conversions exact
}

// Coefficients of one entry; false if a coefficient is not finite.
template <int K>
__device__ __forceinline__ bool entry_coeffs(double r, double s, double b, bool normalise, uint16_t *c)
{
    double norm = 1.0;
    if (normalise) {
        double a = 1.0, t = 0.0;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            t += fabs(a);
            a *= r;
        }
        norm = t;
    }
    double pw = 1.0;
    bool ok = true;
#pragma unroll
    for (int i = 0; i < K; ++i) {
        const double v = (s * pw) / norm + b;
        c[i] = f64_to_f16_rne(v);
        ok = ok && (c[i] & 0x7c00u) != 0x7c00u;
        pw *= r;
    }
    return ok;
}

template <int K>
__device__ __forceinline__ void subset_sums(const uint16_t *c, double *sums)
{
    double cv[K];
#pragma unroll
    for (int i = 0; i < K; ++i)
        cv[i] = f16_bits_to_double(c[i]);
#pragma unroll
    for (int p = 0; p < (1 << K); ++p) {
        double t = 0.0;
#pragma unroll
        for (int i = 0; i < K; ++i)
            if ((p >> i) & 1)
                t += cv[i];
        sums[p] = t;
    }
}

// Nearest subset sum of x: pattern index and the signed difference x - sum.
template <int K>
__device__ __forceinline__ int nearest(const double *sums, double x, double &diff)
{
    int best = 0;
    double bd = x - sums[0];
#pragma unroll
    for (int p = 1; p < (1 << K); ++p) {
        const double d = x - sums[p];
        if (fabs(d) < fabs(bd)) {
            bd = d;
            best = p;
        }
    }
    diff = bd;
    return best;
}

// Smallest squared distance from x to a subset sum: the same value as the
// square of the nearest difference (the rounded square is monotone in |d|),
// without tracking which sum it was.
template <int K>
__device__ __forceinline__ double nearest_sq(const double *sums, double x)
{
    double d = x - sums[0];
    double m = d * d;
#pragma unroll
    for (int p = 1; p < (1 << K); ++p) {
        d = x - sums[p];
        m = fmin(m, d * d);
    }
    return m;
}

constexpr int ENC_CHUNK = 16;  // elements between pruning checks

__device__ __forceinline__ double wave_min_f64(double v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v = fmin(v, __shfl_xor(v, off));
    return v;
}

template <int K>
__device__ __forceinline__ double entry_mse(const double *D, const double *sums)
{
    double err = 0.0;
    for (int j = 0; j < GROUP; ++j) {
        err += nearest_sq<K>(sums, D[j]);
    }
    return err / (double)GROUP;
}

struct EncodeArgs {
    const float *W;
    uint32_t *planes;  // canonical [O][G][K][4]
    uint16_t *coeffs;  // canonical [O][G][K]
    double *mse;       // [O][G] or null
    int O, I;
    int n_ratio1, n_ratio2, n_scale, n_bias, normalise;
};

// A wavefront's LDS for one group: the group's values (read as broadcasts)
// and the search's exchange slots.
struct EncodeLds {
    double D[GROUP];
    double best_mse_l[ENC_THREADS];
    int best_e_l[ENC_THREADS];
    double q_pair[2];
};

template <int K>
struct GroupChoice {
    uint16_t c[K];
    double mse;
    int entry;  // index in the grid, -1 for the no-admissible-entry fallback
};

__device__ __forceinline__ int wave_min_int(int v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v = min(v, __shfl_xor(v, off));
    return v;
}

// Algorithm 1 over the group in L.D (d0, d1: the lane's elements lane and
// lane + 64).  Every lane returns the same choice.
template <int K>
__device__ GroupChoice<K> search_group(const EncodeArgs &a, EncodeLds &L, double d0, double d1)
{
    const int lane = threadIdx.x;
    const double *D = L.D;
    // statistics in element order (every lane, from broadcast reads)
    double mn = D[0], mx = D[0], sum = 0.0;
    for (int j = 0; j < GROUP; ++j) {
        const double v = D[j];
        if (v < mn)
            mn = v;
        if (v > mx)
            mx = v;
        sum += v;
    }
    const double avg = sum / (double)GROUP;

    // sorted positions lo and lo+1 of the linear-interpolation percentile:
    // stable rank of each of the lane's two elements
    const double pos = 0.95 * (double)(GROUP - 1);
    const int lo = (int)floor(pos);
    const double frac = pos - (double)lo;
    {
        int r0 = 0, r1 = 0;
        for (int j = 0; j < GROUP; ++j) {
            const double v = D[j];
            r0 += (v < d0) || (v == d0 && j < lane);
            r1 += (v < d1) || (v == d1 && j < lane + 64);
        }
        if (r0 == lo || r0 == lo + 1)
            L.q_pair[r0 - lo] = d0;
        if (r1 == lo || r1 == lo + 1)
            L.q_pair[r1 - lo] = d1;
    }
    __syncthreads();
    const double q95 = L.q_pair[0] + frac * (L.q_pair[1] - L.q_pair[0]);

    const double s_max = 1.1 * (mx - mn);
    const double s_min = 2.0 * q95;
    const double s_gran = (s_max - s_min) / (double)a.n_scale;
    const double b_max = 2.0 * fabs(avg) / (double)K;
    const double b_min = -b_max;
    const double b_gran = (b_max - b_min) / (double)a.n_bias;
    const double r1_gran = 0.5 / (double)a.n_ratio1;
    const double r2_gran = 1.0 / (double)a.n_ratio2;
    const int per_r = a.n_scale * a.n_bias;
    const int n_entries = (a.n_ratio1 + a.n_ratio2) * per_r;

    auto entry_rsb = [&](int e, double &r, double &s, double &b) {
        const int ir = e / per_r, js = (e / a.n_bias) % a.n_scale, kb = e % a.n_bias;
        r = ir < a.n_ratio1 ? -1.0 + (double)(ir + 1) * r1_gran : -2.0 + (double)(ir - a.n_ratio1) * r2_gran;
        s = s_min + (double)(js + 1) * s_gran;
        b = b_min + (double)kb * b_gran;
    };

    // Pruning (exact): an entry's error sum only grows as elements are added
    // (the terms are >= 0 and rounding is monotone), so once err / n exceeds
    // the smallest MSE any lane has completed, the entry's final MSE is
    // strictly larger than that and it can neither win nor tie; its remaining
    // elements are skipped.  Lanes share their best MSE after every round of
    // 64 entries.
    //
    // Seed for the pruning bound: one round of entries spread over the grid
    // (lane l: ratio l mod |R|, the middle bias, scales spread over the
    // range), each scored over all elements.  Their smallest MSE is an upper
    // bound on the search's minimum (they are entries of the grid), so
    // pruning against it from the first round on stays exact; the search
    // below scores every entry it does not prune, these included, so the
    // result does not depend on the seed.
    double shared_best = __builtin_inf();
    if (n_entries > ENC_THREADS) {
        const int n_r = a.n_ratio1 + a.n_ratio2;
        const int ir = lane % n_r;
        const int per_lane_r = (ENC_THREADS + n_r - 1) / n_r;  // lanes sharing a ratio
        const int js = ((lane / n_r) * a.n_scale + a.n_scale / 2) / per_lane_r % a.n_scale;
        const int e = (ir * a.n_scale + js) * a.n_bias + a.n_bias / 2;
        double r, sc, b;
        entry_rsb(e, r, sc, b);
        uint16_t c[K];
        double mse = __builtin_inf();
        if (sc > 0.0 && entry_coeffs<K>(r, sc, b, a.normalise != 0, c)) {
            double sums[1 << K];
            subset_sums<K>(c, sums);
            mse = entry_mse<K>(D, sums);
        }
        shared_best = wave_min_f64(mse);
    }
    double best_mse = __builtin_inf();
    int best_e = -1;
    for (int e0 = 0; e0 < n_entries; e0 += ENC_THREADS) {
        const int e = e0 + lane;
        bool ok = false;
        double sums[1 << K];
        if (e < n_entries) {
            double r, s, b;
            entry_rsb(e, r, s, b);
            uint16_t c[K];
            ok = s > 0.0 && entry_coeffs<K>(r, s, b, a.normalise != 0, c);
            if (ok)
                subset_sums<K>(c, sums);
        }
        if (ok) {
            double err = 0.0;
            bool pruned = false;
            for (int j0 = 0; j0 < GROUP; j0 += ENC_CHUNK) {
#pragma unroll 4
                for (int j = j0; j < j0 + ENC_CHUNK; ++j) {
                    err += nearest_sq<K>(sums, D[j]);
                }
                if (err / (double)GROUP > shared_best) {
                    pruned = true;
                    break;
                }
            }
            if (!pruned) {
                const double mse = err / (double)GROUP;
                if (mse < best_mse) {
                    best_mse = mse;
                    best_e = e;
                }
            }
        }
        shared_best = wave_min_f64(fmin(shared_best, best_mse));
    }
    L.best_mse_l[lane] = best_mse;
    L.best_e_l[lane] = best_e;
    __syncthreads();
    // smallest error, lowest entry index among equal errors
    double m = __builtin_inf();
    int be = -1;
    for (int l = 0; l < ENC_THREADS; ++l) {
        const int e = L.best_e_l[l];
        const double v = L.best_mse_l[l];
        if (e >= 0 && (be < 0 || v < m || (v == m && e < be))) {
            m = v;
            be = e;
        }
    }

    GroupChoice<K> out;
    if (be >= 0) {
        double r, s, b;
        entry_rsb(be, r, s, b);
        entry_coeffs<K>(r, s, b, a.normalise != 0, out.c);
    } else {  // no admissible entry
        out.c[0] = f64_to_f16_rne(avg);
#pragma unroll
        for (int i = 1; i < K; ++i)
            out.c[i] = 0;
        double sums[1 << K];
        subset_sums<K>(out.c, sums);
        m = entry_mse<K>(D, sums);
    }
    out.mse = m;
    out.entry = be;
    return out;
}

// The bitvector assignment for coefficient set c (each of the lane's two
// elements takes the pattern of its nearest subset sum) and the group's
// stores: plane i by lane i, the coefficients, the MSE by lane 0.
template <int K>
__device__ __forceinline__ void store_group(const EncodeArgs &a, size_t grp, const uint16_t *c, double d0,
                                            double d1, double mse)
{
    const int lane = threadIdx.x;
    double sums[1 << K];
    subset_sums<K>(c, sums);
    double dd;
    const int p0 = nearest<K>(sums, d0, dd), p1 = nearest<K>(sums, d1, dd);
#pragma unroll
    for (int i = 0; i < K; ++i) {
        const uint64_t m0 = __ballot((p0 >> i) & 1), m1 = __ballot((p1 >> i) & 1);
        if (lane == i) {
            uint32_t *pl = a.planes + (grp * K + i) * 4;
            *(uint4 *)pl = make_uint4((uint32_t)m0, (uint32_t)(m0 >> 32), (uint32_t)m1, (uint32_t)(m1 >> 32));
            a.coeffs[grp * K + i] = c[i];
        }
    }
    if (lane == 0 && a.mse)
        a.mse[grp] = mse;
}

template <int K>
__global__ void __launch_bounds__(ENC_THREADS) encode_kernel(EncodeArgs a)
{
    __shared__ EncodeLds L;
    const int lane = threadIdx.x;
    const int G = a.I / GROUP;
    const size_t grp = blockIdx.x;
    const size_t o = grp / G, g = grp % G;
    const float *src = a.W + o * (size_t)a.I + g * GROUP;

    const double d0 = (double)src[lane], d1 = (double)src[lane + 64];
    L.D[lane] = d0;
    L.D[lane + 64] = d1;
    __syncthreads();
    const GroupChoice<K> r = search_group<K>(a, L, d0, d1);
    store_group<K>(a, grp, r.c, d0, d1, r.mse);
}

// The encoder with the cache of Sec. 4.2 (last paragraph and its footnote):
// one wavefront per row, its groups in index order.  Lane s holds cache slot
// s (a coefficient set the full search chose for one of the row's last
// `slots` searched groups, and that group's insertion number; the oldest set
// is replaced first).  For each group every held set is scored with the
// search's MSE (one set per lane, the elements in order); the smallest --
// the oldest among equal ones -- is taken if it is strictly below the mean
// MSE of the row's earlier groups (binary64 sum in group order over their
// count), otherwise the full search runs and its choice enters the cache
// (the no-admissible-entry fallback does not).  The first group of a row
// always searches; with slots = 0 the result is the plain encoder's.
template <int K>
__global__ void __launch_bounds__(ENC_THREADS) encode_cached_kernel(EncodeArgs a, int slots, uint8_t *hits)
{
    __shared__ EncodeLds L;
    const int lane = threadIdx.x;
    const int G = a.I / GROUP;
    const size_t o = blockIdx.x;
    uint16_t cs[K];  // this lane's cached set
#pragma unroll
    for (int i = 0; i < K; ++i)
        cs[i] = 0;
    int seq = INT_MAX;             // its insertion number
    int n_cached = 0, n_ins = 0;   // wavefront-uniform
    double mse_sum = 0.0;          // wavefront-uniform
    for (int g = 0; g < G; ++g) {
        const size_t grp = o * G + g;
        const float *src = a.W + o * (size_t)a.I + (size_t)g * GROUP;
        const double d0 = (double)src[lane], d1 = (double)src[lane + 64];
        __syncthreads();  // the previous group's reads of L are done
        L.D[lane] = d0;
        L.D[lane + 64] = d1;
        __syncthreads();
        bool hit = false;
        uint16_t c[K];
        double mse = 0.0;
        if (g > 0 && n_cached > 0) {
            const double avg = mse_sum / (double)g;
            double m = __builtin_inf();
            if (lane < n_cached) {
                double sums[1 << K];
                subset_sums<K>(cs, sums);
                m = entry_mse<K>(L.D, sums);
            }
            const double best = wave_min_f64(m);
            if (best < avg) {  // wavefront-uniform
                const int oldest = wave_min_int(lane < n_cached && m == best ? seq : INT_MAX);
                const int wl = __ffsll((unsigned long long)__ballot(lane < n_cached && seq == oldest)) - 1;
#pragma unroll
                for (int i = 0; i < K; ++i)
                    c[i] = (uint16_t)__shfl((int)cs[i], wl);
                mse = best;
                hit = true;
            }
        }
        if (!hit) {
            const GroupChoice<K> r = search_group<K>(a, L, d0, d1);
#pragma unroll
            for (int i = 0; i < K; ++i)
                c[i] = r.c[i];
            mse = r.mse;
            if (r.entry >= 0 && slots > 0) {
                if (lane == n_ins % slots) {
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        cs[i] = c[i];
                    seq = n_ins;
                }
                ++n_ins;
                n_cached = min(n_cached + 1, slots);
            }
        }
        store_group<K>(a, grp, c, d0, d1, mse);
        if (lane == 0 && hits)
            hits[grp] = hit ? 1 : 0;
        mse_sum += mse;
    }
}

int launch_encode(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                  int normalise, uint32_t *planes, uint16_t *coeffs, double *mse, hipStream_t stream)
{
    EncodeArgs a = {W, planes, coeffs, mse, O, I, n_ratio1, n_ratio2, n_scale, n_bias, normalise};
    const size_t groups = (size_t)O * (I / GROUP);
    const void *fn = k == 4   ? (const void *)encode_kernel<4>
                     : k == 3 ? (const void *)encode_kernel<3>
                     : k == 2 ? (const void *)encode_kernel<2>
                              : (const void *)encode_kernel<1>;
    void *args[] = {&a};
    return launch_kernel(fn, dim3((unsigned)groups), dim3(ENC_THREADS), 0, stream, args);
}

int launch_encode_cached(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                         int normalise, int slots, uint32_t *planes, uint16_t *coeffs, double *mse, uint8_t *hits,
                         hipStream_t stream)
{
    EncodeArgs a = {W, planes, coeffs, mse, O, I, n_ratio1, n_ratio2, n_scale, n_bias, normalise};
    const void *fn = k == 4   ? (const void *)encode_cached_kernel<4>
                     : k == 3 ? (const void *)encode_cached_kernel<3>
                     : k == 2 ? (const void *)encode_cached_kernel<2>
                              : (const void *)encode_cached_kernel<1>;
    void *args[] = {&a, &slots, &hits};
    return launch_kernel(fn, dim3((unsigned)O), dim3(ENC_THREADS), 0, stream, args);
}

}  // namespace sbvr
