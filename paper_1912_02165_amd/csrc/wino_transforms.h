// Winograd F(m x m, 3 x 3) transform matrices and their application, for the
// GPU kernels.
//
// The transformed convolution of Sec. 2.1, Eq. 3 needs three matrices the paper
// does not print: A^T (m x T), G (T x 3) and B^T (T x T), T = m + 2.  They are
// built here at compile time, in exact rational arithmetic, by the Toom-Cook
// construction: choose T - 1 finite points p_j plus the point at infinity; then
//   A^T[i][j] = p_j^i                        (infinity column: [i == m-1])
//   G[j][u]   = p_j^u / prod_{l!=j}(p_j - p_l) (infinity row: [u == 2])
//   B^T[j][a] = coefficient of x^a in prod_{l!=j}(x - p_l)
//               (infinity row: coefficients of prod_l (x - p_l)).
// Points, in frequency order: F(2): 0, 1, -1; F(4): 0, +-1, +-2;
// F(5): +-1, +-2, +-1/2 (no 0: T = 7 has an even number of finite points);
// F(6): 0, +-1, +-2, +-1/2; F(7): +-1, +-2, +-1/2, +-1/4 (T = 9, no 0).
//
// Because the finite points are (+p, -p) pairs (after 0 for even T), the B^T rows
// of a pair are one polynomial at x and -x: they agree on even coefficients and
// differ in sign on odd ones (and are negated once more for odd T, whose rows
// have odd degree), and the A^T columns of a pair differ by (-1)^i.  The 1D
// transforms below use that to share work between the two rows (even part +-
// odd part).  Every coefficient is a compile-time constant: zero terms vanish,
// +-1 become adds and subtracts.
#pragma once

namespace wino {

// ---- exact rationals, compile time only --------------------------------------
struct Q {
    long long n = 0, d = 1;
};

constexpr long long gcd_ll(long long a, long long b) {
    a = a < 0 ? -a : a;
    b = b < 0 ? -b : b;
    while (b) {
        long long t = a % b;
        a = b;
        b = t;
    }
    return a;
}

constexpr Q mkq(long long n, long long d = 1) {
    if (d < 0) { n = -n; d = -d; }
    long long g = gcd_ll(n, d);
    if (g == 0) g = 1;
    return Q{n / g, d / g};
}
constexpr Q operator+(Q a, Q b) { return mkq(a.n * b.d + b.n * a.d, a.d * b.d); }
constexpr Q operator-(Q a, Q b) { return mkq(a.n * b.d - b.n * a.d, a.d * b.d); }
constexpr Q operator*(Q a, Q b) { return mkq(a.n * b.n, a.d * b.d); }
constexpr Q operator/(Q a, Q b) { return mkq(a.n * b.d, a.d * b.n); }
constexpr bool operator==(Q a, Q b) { return a.n == b.n && a.d == b.d; }
constexpr float to_float(Q a) { return (float)((double)a.n / (double)a.d); }

constexpr Q point(int m, int j) {
    // 0, 1, -1, 2, -2, 1/2, -1/2, 1/4, -1/4: the first m + 1 for even m, without 0
    // for odd m
    constexpr long long num[9] = {0, 1, -1, 2, -2, 1, -1, 1, -1};
    constexpr long long den[9] = {1, 1, 1, 1, 1, 2, 2, 4, 4};
    const int i = (m % 2 == 1) ? j + 1 : j;
    return mkq(num[i], den[i]);
}

// First row (B^T) / column (A^T) of the (+p, -p) pairs: 1 when 0 is a point (even
// T), else 0; and the extra sign between the B^T rows of a pair.
template <int M>
constexpr int pair0() { return (M % 2 == 0) ? 1 : 0; }
template <int M>
constexpr float pair_sign() { return (M % 2 == 0) ? 1.0f : -1.0f; }

template <int M>
struct Tables {
    static constexpr int T = M + 2;
    static constexpr int P = T - 1;  // finite points
    float at[M][T];
    float g[T][3];
    float bt[T][T];

    constexpr Tables() : at{}, g{}, bt{} {
        Q p[P] = {};
        for (int j = 0; j < P; ++j) p[j] = point(M, j);
        // A^T
        for (int i = 0; i < M; ++i) {
            for (int j = 0; j < P; ++j) {
                Q v = mkq(1);
                for (int e = 0; e < i; ++e) v = v * p[j];
                at[i][j] = to_float(v);
            }
            at[i][P] = (i == M - 1) ? 1.0f : 0.0f;
        }
        // G
        for (int j = 0; j < P; ++j) {
            Q den = mkq(1);
            for (int l = 0; l < P; ++l)
                if (l != j) den = den * (p[j] - p[l]);
            Q pw = mkq(1);
            for (int u = 0; u < 3; ++u) {
                g[j][u] = to_float(pw / den);
                pw = pw * p[j];
            }
        }
        g[P][0] = 0.0f; g[P][1] = 0.0f; g[P][2] = 1.0f;
        // B^T: row j from prod_{l != j}(x - p_l), row P from prod_l (x - p_l)
        for (int j = 0; j <= P; ++j) {
            Q c[T] = {};
            c[0] = mkq(1);
            int deg = 0;
            for (int l = 0; l < P; ++l) {
                if (l == j) continue;
                // c(x) *= (x - p_l)
                for (int e = deg + 1; e >= 1; --e) c[e] = c[e - 1] - c[e] * p[l];
                c[0] = mkq(0) - c[0] * p[l];
                ++deg;
            }
            for (int a = 0; a < T; ++a) bt[j][a] = to_float(c[a]);
        }
    }
};

template <int M>
constexpr bool pair_structure_holds() {
    constexpr Tables<M> tb{};
    constexpr int T = M + 2;
    constexpr float sg = pair_sign<M>();
    for (int j = pair0<M>(); j + 1 < T - 1; j += 2) {
        for (int a = 0; a < T; ++a) {
            float e = tb.bt[j][a], o = tb.bt[j + 1][a];
            if (a % 2 == 0 ? (o != sg * e) : (o != -sg * e)) return false;
        }
        for (int i = 0; i < M; ++i) {
            float e = tb.at[i][j], o = tb.at[i][j + 1];
            if (i % 2 == 0 ? (e != o) : (e != -o)) return false;
        }
    }
    return (T - 1 - pair0<M>()) % 2 == 0;  // every finite point but 0 is paired
}
static_assert(pair_structure_holds<2>() && pair_structure_holds<4>() && pair_structure_holds<5>() &&
                  pair_structure_holds<6>() && pair_structure_holds<7>(),
              "B^T rows / A^T columns of +-p points must pair up");

// acc (op)= c * v with a compile-time coefficient; `first` starts the sum.
__device__ __forceinline__ void mac(float &acc, bool &first, float c, float v) {
    if (c == 0.0f) return;
    if (first) {
        acc = (c == 1.0f) ? v : (c == -1.0f) ? -v : c * v;
        first = false;
    } else {
        acc = (c == 1.0f) ? acc + v : (c == -1.0f) ? acc - v : __builtin_fmaf(c, v, acc);
    }
}

// Sum of the terms (c[a] / sc) * in[a*SI], a = A0, A0 + DA, ... < T, evaluated
// starting with a term whose coefficient is +-1 when there is one, so that the
// chain needs no separate multiply.
template <int T, int SI, int A0, int DA>
__device__ __forceinline__ float dot_unit_first(const float (&c)[T], const float *in, float sc = 1.0f) {
    float acc = 0.f;
    bool first = true;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
        for (int a = A0; a < T; a += DA) {
            const float cf = c[a] / sc;
            const bool unit = cf == 1.0f || cf == -1.0f;
            if ((pass == 0) == unit) mac(acc, first, cf, in[a * SI]);
        }
    }
    return acc;
}

// Per row j of B^T and parity (0: even columns, 1: odd columns): a scale by which
// that half of the row is divided so that its sum starts with a coefficient of
// +-1 (no separate multiply), or 1 if the half already has one or is empty.  Only
// powers of two are used, so scaling is exact in fp32.
template <int M>
struct HalfScale {
    float s[M + 2][2];
    static constexpr bool pow2(float c) {
        if (c <= 0.0f) return false;
        while (c < 1.0f) c *= 2.0f;
        while (c > 1.0f) c *= 0.5f;
        return c == 1.0f;
    }
    constexpr HalfScale() : s{} {
        constexpr int T = M + 2;
        Tables<M> tb{};
        for (int j = 0; j < T; ++j)
            for (int par = 0; par < 2; ++par) {
                bool unit = false, any = false;
                float pick = 1.0f;
                for (int a = par; a < T; a += 2) {
                    const float c = tb.bt[j][a] < 0.0f ? -tb.bt[j][a] : tb.bt[j][a];
                    if (c == 0.0f) continue;
                    any = true;
                    if (c == 1.0f) unit = true;
                    else if (pick == 1.0f && pow2(c)) pick = c;
                }
                s[j][par] = (!any || unit) ? 1.0f : pick;
            }
    }
};

// out[i*SO] = sum_a B^T[i][a] in[a*SI], i, a < T.
template <int M, int SI, int SO>
__device__ __forceinline__ void bt_1d(const float *in, float *out) {
    constexpr Tables<M> tb{};
    constexpr HalfScale<M> hs{};
    constexpr int T = M + 2;
    constexpr bool neg = pair_sign<M>() < 0.0f;
    // p = 0 (even T) and the point at infinity: plain rows
    if constexpr (pair0<M>() == 1) out[0] = dot_unit_first<T, SI, 0, 1>(tb.bt[0], in);
    out[(T - 1) * SO] = dot_unit_first<T, SI, 0, 1>(tb.bt[T - 1], in);
#pragma unroll
    for (int j = pair0<M>(); j + 1 < T - 1; j += 2) {
        // (+p, -p) rows: row j = E + O, row j+1 = +-(E - O) with E, O the sums over
        // its even and odd columns, E = se * e and O = so * o
        const float se = hs.s[j][0], so = hs.s[j][1];
        const float e0 = dot_unit_first<T, SI, 0, 2>(tb.bt[j], in, se);
        const float o0 = dot_unit_first<T, SI, 1, 2>(tb.bt[j], in, so);
        // both halves scaled: apply the even scale by itself (one multiply)
        const float e = (se != 1.0f && so != 1.0f) ? se * e0 : e0;
        const float es = (se != 1.0f && so != 1.0f) ? 1.0f : se;
        if (es == 1.0f && so == 1.0f) {
            out[j * SO] = e + o0;
            out[(j + 1) * SO] = neg ? o0 - e : e - o0;
        } else if (es == 1.0f) {
            out[j * SO] = __builtin_fmaf(so, o0, e);
            out[(j + 1) * SO] = neg ? __builtin_fmaf(so, o0, -e) : __builtin_fmaf(-so, o0, e);
        } else {
            out[j * SO] = __builtin_fmaf(es, e, o0);
            out[(j + 1) * SO] = neg ? __builtin_fmaf(-es, e, o0) : __builtin_fmaf(es, e, -o0);
        }
    }
}

// out[i*SO] = sum_j A^T[i][j] in[j*SI], i < M, j < T.
template <int M, int SI, int SO>
__device__ __forceinline__ void at_1d(const float *in, float *out) {
    constexpr Tables<M> tb{};
    constexpr int T = M + 2;
    constexpr int J0 = pair0<M>();
    constexpr int NP = (T - 1 - J0) / 2;  // number of (+p, -p) pairs
    float s[NP], d[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) {
        s[q] = in[(J0 + 2 * q) * SI] + in[(J0 + 1 + 2 * q) * SI];
        d[q] = in[(J0 + 2 * q) * SI] - in[(J0 + 1 + 2 * q) * SI];
    }
#pragma unroll
    for (int i = 0; i < M; ++i) {
        float acc = 0.f;
        bool first = true;
        if constexpr (J0 == 1) mac(acc, first, tb.at[i][0], in[0]);
#pragma unroll
        for (int q = 0; q < NP; ++q) mac(acc, first, tb.at[i][J0 + 2 * q], (i % 2 == 0) ? s[q] : d[q]);
        mac(acc, first, tb.at[i][T - 1], in[(T - 1) * SI]);
        out[i * SO] = acc;
    }
}

// U = B^T d B for a T x T tile held row-major in d; U row-major, frequency i*T + j.
template <int M>
__device__ __forceinline__ void input_tile_transform(const float *d, float *u) {
    constexpr int T = M + 2;
    float tmp[T * T];
#pragma unroll
    for (int b = 0; b < T; ++b) bt_1d<M, T, T>(d + b, tmp + b);       // columns: B^T d
#pragma unroll
    for (int i = 0; i < T; ++i) bt_1d<M, 1, 1>(tmp + i * T, u + i * T);  // rows: (B^T d) B
}

// U = B^T d B as above, handing each finished group of four consecutive
// frequencies to emit(f4, u0, u1, u2, u3) as soon as its rows are done, so the
// whole T^2 result never has to be live at once.
template <int M, class Emit>
__device__ __forceinline__ void input_tile_transform_emit(const float *d, Emit &&emit) {
    constexpr int T = M + 2;
    float tmp[T * T];
#pragma unroll
    for (int b = 0; b < T; ++b) bt_1d<M, T, T>(d + b, tmp + b);       // columns: B^T d
    float u[T * T];
#pragma unroll
    for (int i = 0; i < T; ++i) {
        bt_1d<M, 1, 1>(tmp + i * T, u + i * T);                        // row i of (B^T d) B
#pragma unroll
        for (int f4 = (i * T) / 4; f4 < ((i + 1) * T) / 4; ++f4)      // float4s completed by row i
            emit(f4, u[4 * f4], u[4 * f4 + 1], u[4 * f4 + 2], u[4 * f4 + 3]);
    }
    // odd T: the last float4 holds the last frequency and three zeros
    if constexpr ((T * T) % 4 == 1) emit((T * T) / 4, u[T * T - 1], 0.0f, 0.0f, 0.0f);
}

// Y = A^T Mm A for a T x T tile Mm (row-major); Y is M x M row-major.
template <int M>
__device__ __forceinline__ void output_tile_transform(const float *mm, float *yv) {
    constexpr int T = M + 2;
    float tmp[M * T];
#pragma unroll
    for (int b = 0; b < T; ++b) at_1d<M, T, T>(mm + b, tmp + b);      // columns: A^T Mm
#pragma unroll
    for (int i = 0; i < M; ++i) at_1d<M, 1, 1>(tmp + i * T, yv + i * M);  // rows: (A^T Mm) A
}

// out[i*SO] = sum_{j in ROWS} A^T[i][j] in[j*SI]: A^T applied to a vector whose
// entries outside the bit set ROWS are zero (a +-p pair is either fully in ROWS
// or fully out).  Used when a tile's frequencies are split between waves: by
// linearity each wave inverse-transforms its own rows and the partial outputs
// add up to the full one.
template <int M, int SI, int SO, unsigned ROWS>
__device__ __forceinline__ void at_1d_rows(const float *in, float *out) {
    constexpr Tables<M> tb{};
    constexpr int T = M + 2;
    constexpr int J0 = pair0<M>();
    constexpr int NP = (T - 1 - J0) / 2;
    float s[NP], d[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) {
        if ((ROWS >> (J0 + 2 * q)) & 1u) {
            s[q] = in[(J0 + 2 * q) * SI] + in[(J0 + 1 + 2 * q) * SI];
            d[q] = in[(J0 + 2 * q) * SI] - in[(J0 + 1 + 2 * q) * SI];
        }
    }
#pragma unroll
    for (int i = 0; i < M; ++i) {
        float acc = 0.f;
        bool first = true;
        if (J0 == 1 && (ROWS & 1u)) mac(acc, first, tb.at[i][0], in[0]);
#pragma unroll
        for (int q = 0; q < NP; ++q)
            if ((ROWS >> (J0 + 2 * q)) & 1u) mac(acc, first, tb.at[i][J0 + 2 * q], (i % 2 == 0) ? s[q] : d[q]);
        if ((ROWS >> (T - 1)) & 1u) mac(acc, first, tb.at[i][T - 1], in[(T - 1) * SI]);
        out[i * SO] = first ? 0.0f : acc;
    }
}

template <int M, unsigned ROWS>
constexpr bool rows_pair_closed() {
    constexpr int T = M + 2;
    for (int j = pair0<M>(); j + 1 < T - 1; j += 2)
        if (((ROWS >> j) & 1u) != ((ROWS >> (j + 1)) & 1u)) return false;
    return true;
}

// Partial output tile: Y_part = A^T Mm_rows A, where only the transform-domain
// rows in ROWS of Mm (row-major T x T) are used.
template <int M, unsigned ROWS>
__device__ __forceinline__ void output_tile_transform_rows(const float *mm, float *yv) {
    static_assert(rows_pair_closed<M, ROWS>(), "row set must hold whole +-p pairs");
    constexpr int T = M + 2;
    float tmp[M * T];
#pragma unroll
    for (int b = 0; b < T; ++b) at_1d_rows<M, T, T, ROWS>(mm + b, tmp + b);
#pragma unroll
    for (int i = 0; i < M; ++i) at_1d<M, 1, 1>(tmp + i * T, yv + i * M);
}

// W' = G g G^T for a 3 x 3 kernel g (row-major); W' is T x T row-major.
template <int M>
__device__ __forceinline__ void kernel_tile_transform(const float *g, float *wt) {
    constexpr Tables<M> tb{};
    constexpr int T = M + 2;
    float tmp[T * 3];
#pragma unroll
    for (int i = 0; i < T; ++i)
#pragma unroll
        for (int v = 0; v < 3; ++v) {
            float acc = 0.f;
            bool first = true;
#pragma unroll
            for (int u = 0; u < 3; ++u) mac(acc, first, tb.g[i][u], g[u * 3 + v]);
            tmp[i * 3 + v] = first ? 0.f : acc;
        }
#pragma unroll
    for (int i = 0; i < T; ++i)
#pragma unroll
        for (int j = 0; j < T; ++j) {
            float acc = 0.f;
            bool first = true;
#pragma unroll
            for (int v = 0; v < 3; ++v) mac(acc, first, tb.g[j][v], tmp[i * 3 + v]);
            wt[i * T + j] = first ? 0.f : acc;
        }
}

}  // namespace wino
