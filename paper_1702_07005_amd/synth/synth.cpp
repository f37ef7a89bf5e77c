// synth.cpp -- seeded synthetic sparse inputs shaped like the workloads of
// "Large-Scale Stochastic Learning using GPUs" (arXiv 1702.07005): a dense Gaussian
// regression problem, a uniform-random sparse regression problem, a text-like
// matrix with Zipf column popularity (stand-in for the webspam sample of Sec. III-D)
// and a click-log-like one-hot matrix (stand-in for one worker's share of the criteo
// sample of Sec. V-B).
//
// This module only makes inputs: it holds none of the coordinate-descent arithmetic
// and is shared by the HIP path's tests/benchmark and by the oracle's tests.
//
// Determinism: every row is drawn from its own counter-based stream keyed by
// (seed, stream tag, row), so the output is identical for any thread count.
// Generators used:
//   * SplitMix64 (Steele, Lea, Flood 2014) as the counter-based uniform source;
//   * Box-Muller for normals;
//   * rejection-inversion for Zipf ranks (Hoermann & Derflinger 1996), O(1) memory;
//   * geometric skipping for Bernoulli(p) column selection;
//   * affine bijections x -> (a x + b) mod n, gcd(a, n) = 1, to scatter Zipf ranks.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <numeric>
#include <vector>
#include <omp.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ULL;

inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

// Stream tags keep the different draws of one row independent.
enum : uint64_t {
    TAG_ROW = 0x524F5753ULL,     // per-row stream (columns, values, label noise)
    TAG_XSTAR = 0x58535452ULL,   // dense planted model x*
    TAG_HSEL = 0x4853454CULL,    // hyperplane support selection
    TAG_HVAL = 0x4856414CULL,    // hyperplane values
    TAG_PERM = 0x5045524DULL,    // rank -> column bijections
};

inline uint64_t key_of(uint64_t seed, uint64_t tag, uint64_t i) {
    return mix64(mix64(seed ^ mix64(tag)) + kGamma * (i + 1));
}

inline double u01(uint64_t x) {  // (0, 1), never 0 or 1
    return ((double)(x >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

struct Stream {
    uint64_t s;
    bool have = false;
    double spare = 0.0;
    explicit Stream(uint64_t key) : s(key) {}
    uint64_t next() { s += kGamma; return mix64(s); }
    double uniform() { return u01(next()); }
    double normal() {
        if (have) { have = false; return spare; }
        double r = std::sqrt(-2.0 * std::log(uniform()));
        double t = 6.283185307179586476925 * uniform();
        spare = r * std::sin(t);
        have = true;
        return r * std::cos(t);
    }
};

// A normal deviate that is a pure function of a key (for per-feature planted values).
inline double keyed_normal(uint64_t key) {
    double u1 = u01(mix64(key + kGamma));
    double u2 = u01(mix64(key + 2 * kGamma));
    return std::sqrt(-2.0 * std::log(u1)) * std::cos(6.283185307179586476925 * u2);
}

// Zipf(s) on {1..n} by rejection-inversion (Hoermann & Derflinger 1996).
struct Zipf {
    double s = 1.0, n = 1.0, hx1 = 0.0, hn = 0.0, sc = 0.0;
    static double helper1(double x) {  // log1p(x)/x
        return std::fabs(x) > 1e-8 ? std::log1p(x) / x : 1.0 - x * (0.5 - x * (1.0 / 3.0 - 0.25 * x));
    }
    static double helper2(double x) {  // expm1(x)/x
        return std::fabs(x) > 1e-8 ? std::expm1(x) / x : 1.0 + x * 0.5 * (1.0 + x * (1.0 / 3.0) * (1.0 + 0.25 * x));
    }
    double H(double x) const { double lx = std::log(x); return helper2((1.0 - s) * lx) * lx; }
    double h(double x) const { return std::exp(-s * std::log(x)); }
    double Hinv(double x) const {
        double t = x * (1.0 - s);
        if (t < -1.0) t = -1.0;
        return std::exp(helper1(t) * x);
    }
    Zipf() = default;
    Zipf(double s_, int64_t n_) : s(s_), n((double)n_) {
        hx1 = H(1.5) - 1.0;
        hn = H(n + 0.5);
        sc = 2.0 - Hinv(H(2.5) - h(2.0));
    }
    int64_t sample(Stream& st) const {
        for (;;) {
            double u = hn + st.uniform() * (hx1 - hn);
            double x = Hinv(u);
            int64_t k = (int64_t)(x + 0.5);
            if (k < 1) k = 1;
            if ((double)k > n) k = (int64_t)n;
            if ((double)k - x <= sc || u >= H((double)k + 0.5) - h((double)k)) return k;
        }
    }
};

struct Affine {  // x -> (a x + b) mod n, a bijection of [0, n) when gcd(a, n) = 1
    uint64_t a = 1, b = 0, n = 1;
    Affine() = default;
    Affine(uint64_t key, uint64_t n_) : n(n_) {
        if (n <= 1) { a = 1; b = 0; return; }
        a = (mix64(key) % n) | 1;
        while (std::gcd(a, n) != 1) a = (a + 2) % n == 0 ? 1 : (a + 2) % n;
        b = mix64(key + kGamma) % n;
    }
    uint64_t operator()(uint64_t x) const {
        unsigned __int128 t = (unsigned __int128)a * x + b;
        return (uint64_t)(t % n);
    }
};

}  // namespace

extern "C" {

// kind: 0 dense Gaussian rows (all n_cols columns, values N(0,1));
//       1 Bernoulli(density) columns per row, values N(0,1);
//       2 text-like: row_nnz distinct columns drawn Zipf(zipf_s) over ranks, values exp(N(0,1)),
//         labels = sign of a sparse random hyperplane with a fraction `flip` of them flipped;
//       3 click-like: row_nnz fields, field f has cardinality proportional to f^-zipf_s
//         (summing to n_cols), one Zipf(zipf_s) value per field, binary values,
//         labels +1 with probability pos_rate, else -1.
// Kinds 0/1 label with y = x.x* + noise * N(0,1), x* ~ N(0,1) per feature.
// normalize != 0 scales every non-empty row to unit L2 norm.
typedef struct {
    int32_t kind;
    int32_t normalize;
    uint64_t seed;
    int64_t n_rows;
    int64_t n_cols;
    double density;
    int32_t row_nnz;
    int32_t pad_;
    double zipf_s;
    double noise;
    double hyper_frac;
    double flip;
    double pos_rate;
} synth_spec;

}  // extern "C"

namespace {

struct Fields {  // kind 3 layout
    std::vector<int64_t> card, offset;
    std::vector<Zipf> zipf;
    std::vector<Affine> perm;
};

Fields make_fields(const synth_spec& sp) {
    Fields F;
    int nf = sp.row_nnz;
    std::vector<double> w(nf);
    double W = 0.0;
    for (int f = 0; f < nf; ++f) { w[f] = std::pow((double)(f + 1), -sp.zipf_s); W += w[f]; }
    F.card.resize(nf);
    int64_t used = 0;
    for (int f = 0; f < nf; ++f) {
        int64_t c = (int64_t)std::floor((double)sp.n_cols * w[f] / W);
        if (c < 1) c = 1;
        F.card[f] = c;
        used += c;
    }
    // Hand the rounding remainder to the largest field (keeps the sum exactly n_cols).
    F.card[0] += sp.n_cols - used;
    F.offset.resize(nf);
    int64_t off = 0;
    for (int f = 0; f < nf; ++f) { F.offset[f] = off; off += F.card[f]; }
    F.zipf.resize(nf);
    F.perm.resize(nf);
    for (int f = 0; f < nf; ++f) {
        F.zipf[f] = Zipf(sp.zipf_s, F.card[f]);
        F.perm[f] = Affine(key_of(sp.seed, TAG_PERM, (uint64_t)f + 1), (uint64_t)F.card[f]);
    }
    return F;
}

int check(const synth_spec* sp) {
    if (!sp || sp->n_rows < 0 || sp->n_cols < 1 || sp->n_cols > 2147483647LL) return -1;
    if (sp->kind < 0 || sp->kind > 3) return -1;
    if (sp->kind == 1 && !(sp->density > 0.0 && sp->density <= 1.0)) return -1;
    if ((sp->kind == 2 || sp->kind == 3) && (sp->row_nnz < 1 || sp->zipf_s <= 0.0 || sp->zipf_s == 1.0)) return -1;
    if (sp->kind == 2 && sp->row_nnz > sp->n_cols) return -1;
    if (sp->kind == 3 && sp->row_nnz > sp->n_cols) return -1;
    return 0;
}

// Columns of one kind-1 row by geometric skipping over Bernoulli(p) trials.
template <class Emit>
void bernoulli_row(Stream& st, int64_t n_cols, double p, Emit emit) {
    if (p >= 1.0) { for (int64_t c = 0; c < n_cols; ++c) emit(c); return; }
    double lq = std::log1p(-p);
    int64_t c = -1;
    for (;;) {
        double g = std::floor(std::log(st.uniform()) / lq);
        if (g >= (double)n_cols) break;
        c += 1 + (int64_t)g;
        if (c >= n_cols) break;
        emit(c);
    }
}

}  // namespace

extern "C" {

// Pass 1: the number of stored entries of every row.
int synth_row_lengths(const synth_spec* sp, int64_t* len, int n_threads) {
    if (check(sp)) return -1;
    const synth_spec S = *sp;
    if (S.kind == 0) { for (int64_t r = 0; r < S.n_rows; ++r) len[r] = S.n_cols; return 0; }
    if (S.kind == 2 || S.kind == 3) { for (int64_t r = 0; r < S.n_rows; ++r) len[r] = S.row_nnz; return 0; }
#pragma omp parallel for schedule(dynamic, 1024) num_threads(n_threads)
    for (int64_t r = 0; r < S.n_rows; ++r) {
        Stream st(key_of(S.seed, TAG_ROW, (uint64_t)r));
        int64_t k = 0;
        bernoulli_row(st, S.n_cols, S.density, [&](int64_t) { ++k; });
        len[r] = k;
    }
    return 0;
}

// Pass 2: fill CSR (row_ptr given, from pass 1) and the labels.
int synth_fill(const synth_spec* sp, const int64_t* row_ptr, int32_t* col_idx, float* val, float* y,
               int n_threads) {
    if (check(sp)) return -1;
    const synth_spec S = *sp;
    Fields F;
    if (S.kind == 3) F = make_fields(S);
    Zipf z2;
    Affine a2;
    if (S.kind == 2) {
        z2 = Zipf(S.zipf_s, S.n_cols);
        a2 = Affine(key_of(S.seed, TAG_PERM, 0), (uint64_t)S.n_cols);
    }
    const uint64_t kx = key_of(S.seed, TAG_XSTAR, 0);
    const uint64_t khs = key_of(S.seed, TAG_HSEL, 0);
    const uint64_t khv = key_of(S.seed, TAG_HVAL, 0);
    std::atomic<int> bad{0};

#pragma omp parallel num_threads(n_threads)
    {
        std::vector<int64_t> cols;
        std::vector<double> vals;
        // kind 2: open-addressing set of drawn ranks, cleared by generation stamps.
        size_t cap = 16;
        if (S.kind == 2) while (cap < (size_t)S.row_nnz * 4) cap <<= 1;
        std::vector<int64_t> slot(S.kind == 2 ? cap : 0);
        std::vector<uint32_t> stamp(S.kind == 2 ? cap : 0, 0);
        uint32_t gen = 0;

#pragma omp for schedule(dynamic, 64)
        for (int64_t r = 0; r < S.n_rows; ++r) {
            Stream st(key_of(S.seed, TAG_ROW, (uint64_t)r));
            cols.clear();
            vals.clear();
            double label = 0.0;
            if (S.kind == 0) {
                for (int64_t c = 0; c < S.n_cols; ++c) { cols.push_back(c); vals.push_back(st.normal()); }
            } else if (S.kind == 1) {
                bernoulli_row(st, S.n_cols, S.density, [&](int64_t c) { cols.push_back(c); });
                for (size_t k = 0; k < cols.size(); ++k) vals.push_back(st.normal());
            } else if (S.kind == 2) {
                ++gen;
                if (gen == 0) { std::fill(stamp.begin(), stamp.end(), 0); gen = 1; }
                const size_t m = cap - 1;
                while ((int)cols.size() < S.row_nnz) {
                    int64_t rank = z2.sample(st);
                    size_t hsh = (size_t)mix64((uint64_t)rank) & m;
                    bool dup = false;
                    while (stamp[hsh] == gen) {
                        if (slot[hsh] == rank) { dup = true; break; }
                        hsh = (hsh + 1) & m;
                    }
                    if (dup) continue;
                    stamp[hsh] = gen;
                    slot[hsh] = rank;
                    cols.push_back((int64_t)a2((uint64_t)(rank - 1)));
                }
                std::sort(cols.begin(), cols.end());
                for (size_t k = 0; k < cols.size(); ++k) vals.push_back(std::exp(st.normal()));
            } else {
                for (int f = 0; f < S.row_nnz; ++f) {
                    int64_t rank = F.zipf[f].sample(st);
                    cols.push_back(F.offset[f] + (int64_t)F.perm[f]((uint64_t)(rank - 1)));
                    vals.push_back(1.0);
                }
            }
            if (S.normalize) {
                double s = 0.0;
                for (double v : vals) s += v * v;
                if (s > 0.0) { s = 1.0 / std::sqrt(s); for (double& v : vals) v *= s; }
            }
            const int64_t base = row_ptr[r];
            if (row_ptr[r + 1] - base != (int64_t)cols.size()) { bad = 1; continue; }
            for (size_t k = 0; k < cols.size(); ++k) {
                col_idx[base + (int64_t)k] = (int32_t)cols[k];
                val[base + (int64_t)k] = (float)vals[k];
            }
            if (S.kind == 0 || S.kind == 1) {
                double d = 0.0;
                for (size_t k = 0; k < cols.size(); ++k)
                    d += (double)(float)vals[k] * keyed_normal(kx + kGamma * 3 * (uint64_t)cols[k]);
                label = d + S.noise * st.normal();
            } else if (S.kind == 2) {
                double d = 0.0;
                for (size_t k = 0; k < cols.size(); ++k) {
                    uint64_t c = (uint64_t)cols[k];
                    if (u01(mix64(khs + kGamma * c)) < S.hyper_frac)
                        d += (double)(float)vals[k] * keyed_normal(khv + kGamma * 3 * c);
                }
                label = d >= 0.0 ? 1.0 : -1.0;
                if (st.uniform() < S.flip) label = -label;
            } else {
                label = st.uniform() < S.pos_rate ? 1.0 : -1.0;
            }
            y[r] = (float)label;
        }
    }
    return bad ? -2 : 0;
}

// The field layout of kind 3 (cardinalities and column offsets), for inspection.
int synth_fields(const synth_spec* sp, int64_t* card, int64_t* offset) {
    if (check(sp) || sp->kind != 3) return -1;
    Fields F = make_fields(*sp);
    for (int f = 0; f < sp->row_nnz; ++f) { card[f] = F.card[f]; offset[f] = F.offset[f]; }
    return 0;
}

// Raw Zipf draws (for distribution checks of the sampler).
int synth_zipf_draws(double s, int64_t n, uint64_t seed, int64_t count, int64_t* out) {
    if (s <= 0.0 || s == 1.0 || n < 1) return -1;
    Zipf z(s, n);
    Stream st(key_of(seed, TAG_ROW, 0));
    for (int64_t i = 0; i < count; ++i) out[i] = z.sample(st);
    return 0;
}

// CSR -> CSC transpose, rows sorted inside every column.  Deterministic: thread t owns
// a contiguous block of rows and gets its own slice of every column's range.
int synth_csr_to_csc(int64_t n_rows, int64_t n_cols, const int64_t* row_ptr, const int32_t* col_idx,
                     const float* val, int64_t* col_ptr, int32_t* row_idx, float* cval, int n_threads) {
    if (n_threads < 1) n_threads = 1;
    const int T = n_threads;
    const int64_t nnz = row_ptr[n_rows];
    std::vector<int64_t> rb(T + 1);
    for (int t = 0; t <= T; ++t) {
        int64_t target = nnz / T * t + std::min<int64_t>(t, nnz % T);
        rb[t] = std::lower_bound(row_ptr, row_ptr + n_rows + 1, target) - row_ptr;
        if (rb[t] > n_rows) rb[t] = n_rows;
    }
    rb[0] = 0;
    rb[T] = n_rows;
    for (int t = 1; t <= T; ++t) if (rb[t] < rb[t - 1]) rb[t] = rb[t - 1];
    std::vector<std::vector<int64_t>> cnt(T);
    std::atomic<int> bad{0};
#pragma omp parallel num_threads(T)
    {
        int t = omp_get_thread_num();
        cnt[t].assign((size_t)n_cols, 0);
        for (int64_t r = rb[t]; r < rb[t + 1]; ++r)
            for (int64_t k = row_ptr[r]; k < row_ptr[r + 1]; ++k) {
                int32_t c = col_idx[k];
                if (c < 0 || c >= n_cols) { bad = 1; continue; }
                ++cnt[t][(size_t)c];
            }
    }
    if (bad) return -1;
    // col_ptr and per-thread cursors (cnt[t][c] becomes thread t's write position in column c).
    col_ptr[0] = 0;
    for (int64_t c = 0; c < n_cols; ++c) {
        int64_t pos = col_ptr[c];
        for (int t = 0; t < T; ++t) { int64_t n = cnt[t][(size_t)c]; cnt[t][(size_t)c] = pos; pos += n; }
        col_ptr[c + 1] = pos;
    }
#pragma omp parallel num_threads(T)
    {
        int t = omp_get_thread_num();
        std::vector<int64_t>& cur = cnt[t];
        for (int64_t r = rb[t]; r < rb[t + 1]; ++r)
            for (int64_t k = row_ptr[r]; k < row_ptr[r + 1]; ++k) {
                int64_t p = cur[(size_t)col_idx[k]]++;
                row_idx[p] = (int32_t)r;
                cval[p] = val[k];
            }
    }
    return 0;
}

}  // extern "C"
