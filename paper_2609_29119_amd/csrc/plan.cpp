// Host plan builder: band layout, windows, dual windows, routing weights,
// ownership of bins for the atomics-free overlap-add, FFT plans, twiddles and
// Bluestein tables. All values are computed in fp64 and rounded once to fp32.
#include "plan.hpp"

#include <algorithm>
#include <cmath>
#include <complex>
#include <limits>
#include <map>

#include "../../include/nsgcqt.h"

namespace nsg {

namespace {

using cd = std::complex<double>;
constexpr double kPi = 3.14159265358979323846264338327950288;

int64_t align256(int64_t b) { return (b + 255) / 256 * 256; }

// exp(-2 pi i t / n) with t reduced modulo n first.
cd root(int64_t t, int64_t n) {
    t %= n;
    if (t < 0) t += n;
    const double ang = 2.0 * kPi * static_cast<double>(t) / static_cast<double>(n);
    return cd(std::cos(ang), -std::sin(ang));
}

int smallest_prime_factor(int64_t n) {
    if (n % 2 == 0) return 2;
    for (int64_t p = 3; p * p <= n; p += 2)
        if (n % p == 0) return static_cast<int>(p);
    return static_cast<int>(n);
}

// Forward DFT (eq. 1) of a smooth length in fp64, recursive decimation in
// time. Used only at plan time for the Bluestein kernels.
// Decimation in time by the smallest prime factor of n; w holds
// omega_N^t for t < N, and a length-n subproblem uses its every (N/n)-th entry.
void dft_rec(std::vector<cd>& x, const std::vector<cd>& w) {
    const int64_t n = static_cast<int64_t>(x.size());
    if (n <= 1) return;
    const int64_t N = static_cast<int64_t>(w.size()), step = N / n;
    const int p = smallest_prime_factor(n);
    const int64_t m = n / p;
    std::vector<std::vector<cd>> sub(p, std::vector<cd>(m));
    for (int64_t j = 0; j < m; ++j)
        for (int r = 0; r < p; ++r) sub[r][j] = x[j * p + r];
    for (int r = 0; r < p; ++r) dft_rec(sub[r], w);
    // X_k = sum_r omega_n^{r k} S_r[k mod m], k = q m + j; e tracks r k mod n
    std::fill(x.begin(), x.end(), cd(0.0, 0.0));
    for (int r = 0; r < p; ++r) {
        const std::vector<cd>& sr = sub[r];
        int64_t e = 0;
        for (int64_t q = 0, k = 0; q < p; ++q)
            for (int64_t j = 0; j < m; ++j, ++k) {
                x[k] += sr[j] * w[e * step];
                e += r;
                if (e >= n) e -= n;
            }
    }
}

// In-place DFT in fp64 (mixed radix; the roots are computed once, each with
// its angle reduced exactly).
void host_dft(std::vector<cd>& x) {
    const int64_t n = static_cast<int64_t>(x.size());
    if (n <= 1) return;
    std::vector<cd> w(n);
    for (int64_t t = 0; t < n; ++t) w[t] = root(t, n);
    dft_rec(x, w);
}

void push_c(std::vector<float>& v, cd z) {
    v.push_back(static_cast<float>(z.real()));
    v.push_back(static_cast<float>(z.imag()));
}

}  // namespace

bool factor_radices(int64_t n, std::vector<int>& out, int max_prime) {
    out.clear();
    if (n < 1) return false;
    // prime factors, largest first
    std::vector<int64_t> f;
    int64_t m = n;
    for (int64_t p = 2; p * p <= m; ++p)
        while (m % p == 0) { f.push_back(p); m /= p; }
    if (m > 1) f.push_back(m);
    std::sort(f.rbegin(), f.rend());
    // primes above 16 are stages of their own (runtime radix, up to
    // max_prime); the rest are packed greedily into compile-time radices of
    // at most 16
    std::vector<int64_t> small;
    for (int64_t p : f) {
        if (p > 16) {
            if (p > max_prime) return false;
            out.push_back(static_cast<int>(p));
        } else {
            small.push_back(p);
        }
    }
    while (!small.empty()) {
        int64_t r = small.front();
        small.erase(small.begin());
        for (size_t i = 0; i < small.size();) {
            if (r * small[i] <= 16) {
                r *= small[i];
                small.erase(small.begin() + static_cast<long>(i));
            } else {
                ++i;
            }
        }
        out.push_back(static_cast<int>(r));
    }
    return static_cast<int>(out.size()) <= kMaxStages;
}

namespace {

struct FftRegistry {
    HostPlan& p;
    std::map<int64_t, int> index;
    explicit FftRegistry(HostPlan& plan) : p(plan) {}

    // Index of the FftDesc for length n, creating it (and its twiddles) on
    // first use; -1 if n does not factor into supported radices.
    int get(int64_t n) {
        auto it = index.find(n);
        if (it != index.end()) return it->second;
        std::vector<int> rad;
        if (!factor_radices(n, rad)) return -1;
        FftDesc d{};
        d.n = static_cast<int32_t>(n);
        d.nstages = static_cast<int32_t>(rad.size());
        for (size_t s = 0; s < rad.size(); ++s) d.radix[s] = static_cast<int16_t>(rad[s]);
        d.full = static_cast<int32_t>(p.twpool.size() / 2);
        for (int64_t t = 0; t < n; ++t) push_c(p.twpool, root(t, n));
        int lg = 0;
        while ((int64_t(1) << (2 * lg)) < n) ++lg;
        d.lg = lg;
        d.nhi = static_cast<int32_t>((n + (int64_t(1) << lg) - 1) >> lg);
        for (int64_t i = 0; i < d.nhi; ++i) push_c(p.twpool, root(i << lg, n));
        for (int64_t j = 0; j < (int64_t(1) << lg); ++j) push_c(p.twpool, root(j, n));
        // stage twiddles omega_{Ns R}^{r k} = omega_n^{r k n / (Ns R)}
        d.stw = static_cast<int32_t>(p.twpool.size() / 2);
        int64_t Ns = 1, off = 0;
        for (size_t s = 0; s < rad.size(); ++s) {
            const int64_t R = rad[s];
            d.rcp_ns[s] = static_cast<float>(1.0 / static_cast<double>(Ns));
            d.rcp_h[s] = R > 16 ? static_cast<float>(1.0 / static_cast<double>((R - 1) / 2)) : 0.0f;
            d.stoff[s] = static_cast<int32_t>(off);
            if (s > 0) {
                const int64_t stride = n / (Ns * R);
                for (int64_t k = 0; k < Ns; ++k)
                    for (int64_t r = 1; r < R; ++r) push_c(p.twpool, root(r * k * stride, n));
                off += (R - 1) * Ns;
            }
            Ns *= R;
        }
        d.ntw = static_cast<int32_t>(off);
        p.ffts.push_back(d);
        const int id = static_cast<int>(p.ffts.size()) - 1;
        index[n] = id;
        return id;
    }
};

int fail(std::string& err, int code, const std::string& msg) {
    err = msg;
    return code;
}

// Tiles a four-step pass aims for at least: 2.5 per compute unit of MI355X
// (256 CUs), so that the last round of a persistent pass is not a long tail.
constexpr int64_t kPassTiles = 640;

// Band kernel tiers by transform length: threads and elements per thread.
struct Tier { int max_work, nt, ept; };
constexpr Tier kTiers[] = {{512, 64, 8}, {2048, 256, 8}, {4096, 256, 16}, {8192, 512, 16}, {16384, 1024, 16}};
constexpr int kNumTiers = static_cast<int>(sizeof(kTiers) / sizeof(kTiers[0]));

int tier_of(int64_t n) {
    for (int i = 0; i < kNumTiers; ++i)
        if (n <= kTiers[i].max_work) return i;
    return -1;
}

// log2 of the interleaved sequences per band work item of a length-n
// transform: at most 16, within E elements, no more than the batch needs, and
// 2^lg rows of Z and of coefficients (row_bytes each) within 32-bit offsets.
int seq_lg(int64_t n, int E, int batch, int64_t row_bytes) {
    int lg = 4;
    while (lg > 0 && ((int64_t(1) << lg) * n > E || (1 << (lg - 1)) >= batch ||
                      (int64_t(1) << lg) * row_bytes >= (int64_t(1) << 32)))
        --lg;
    return lg;
}

// True when every prime-radix stage (R > 16) of a length-n transform keeps
// its matrix-core result tiles within the workgroup when 2^lg sequences share
// a workgroup of nt threads.
bool mfma_fits(const std::vector<int>& rad, int64_t n, int lg, int nt) {
    for (int R : rad)
        if (R > 16 && mfma_tiles(static_cast<int>((n / R) << lg), R) > kMfmaTilesPerWave * (nt / 64)) return false;
    return true;
}

// Estimated cost, in SIMD cycles per sequence, of a length-n transform with
// the given radices when 2^lg sequences share a workgroup: about 20 vector
// instructions per point for a compile-time stage; a matrix-core stage costs
// its fold and write passes plus 2 Kb products of 32 cycles per result tile.
double stage_cost(const std::vector<int>& rad, int64_t n, int lg) {
    double c = 0.0;
    for (int R : rad) {
        if (R <= 16) {
            c += 1.25 * static_cast<double>(n);
        } else {
            const int Kb = ((R - 1) / 2 + 3) >> 2;
            const int tiles = mfma_tiles(static_cast<int>((n / R) << lg), R);
            c += 0.9 * static_cast<double>(n) + tiles * Kb * 64.0 / static_cast<double>(1 << lg);
        }
    }
    return c;
}

// Column length n1 of the four-step split n = n1 n2 (n1 <= n2 <= 4096, both
// with a radix plan) used for transforms beyond the largest tier; -1 if none.
int64_t huge_split(int64_t n) {
    int64_t n1 = -1;
    for (int64_t d = 2; d * d <= n; ++d) {
        std::vector<int> r1, r2;
        if (n % d == 0 && n / d <= 4096 && factor_radices(d, r1) && factor_radices(n / d, r2)) n1 = d;
    }
    return n1;
}

// Where a length-n band transform runs: the tier (-1: the four-step
// huge-band path) and the largest interleave at which its prime-radix stages'
// matrix tiles fit that tier's workgroup.
struct BandFit {
    int tier;
    int lg_cap;
    double cost;
};

// Cost of a length-n band transform: in the smallest tier that holds it and
// fits its matrix tiles at some interleave (the largest such interleave up to
// seq_lg for an unbounded batch), or, above the largest tier, in the
// four-step huge-band path; infinite when it cannot run. The choice depends on
// n alone, not on the batch, so every result bit is the same for any batch
// size and position.
BandFit band_fft_fit(int64_t n, int64_t row_bytes) {
    const double inf = std::numeric_limits<double>::infinity();
    std::vector<int> rad;
    if (!factor_radices(n, rad)) return BandFit{-1, 0, inf};
    const int t0 = tier_of(n);
    if (t0 < 0) {
        if (huge_split(n) < 0) return BandFit{-1, 0, inf};
        return BandFit{-1, 0, 2.5 * static_cast<double>(n) * static_cast<double>(rad.size())};
    }
    for (int ti = t0; ti < kNumTiers; ++ti) {
        const Tier& t = kTiers[ti];
        for (int lg = seq_lg(n, t.nt * t.ept, 1 << 30, row_bytes); lg >= 0; --lg)
            if (mfma_fits(rad, n, lg, t.nt)) return BandFit{ti, lg, stage_cost(rad, n, lg)};
    }
    return BandFit{-1, 0, inf};
}

double band_fft_cost(int64_t n, int64_t row_bytes) { return band_fft_fit(n, row_bytes).cost; }

// Bluestein length for a band of length M: among the P >= 2M - 1 (up to a
// quarter longer) whose prime factors are all compile-time radices (2..13),
// the one with the lowest estimated cost of two length-P transforms and the
// three pointwise products; *cost receives that cost.
int64_t bluestein_length(int64_t M, int64_t row_bytes, double* cost) {
    const int64_t lo = 2 * M - 1, hi = lo + lo / 4 + 16;
    int64_t best = -1;
    double best_c = std::numeric_limits<double>::infinity();
    for (int64_t P = lo; P <= hi; ++P) {
        int64_t m = P;
        for (int q : {2, 3, 5, 7, 11, 13})
            while (m % q == 0) m /= q;
        if (m != 1) continue;
        const double c = 2.0 * band_fft_cost(P, row_bytes) + 0.6 * static_cast<double>(P);
        if (c < best_c) {
            best_c = c;
            best = P;
        }
    }
    *cost = best_c;
    return best;
}

}  // namespace

namespace {

// Checks and settings shared by both plan builders.
int begin_plan(HostPlan& p, double fs, int64_t N, int batch, bool sliced, std::string& err) {
    if (!(N >= 4) || (N % 2) != 0)
        return fail(err, NSGCQT_EINVAL, "n_samples must be even and >= 4");
    if (!(fs > 0.0)) return fail(err, NSGCQT_EINVAL, "fs must be > 0");
    if (batch < 1) return fail(err, NSGCQT_EINVAL, "batch must be >= 1");
    if (sliced && (N % 8) != 0)
        return fail(err, NSGCQT_EINVAL, "slice length must be a multiple of 8");
    // the band kernels address a signal's packed spectrum and coefficient row
    // with 32-bit byte offsets
    if (N >= (int64_t(1) << 29))
        return fail(err, NSGCQT_EUNSUPPORTED, "n_samples of 2^29 or more");
    p.fs = fs;
    p.N = N; p.L = N / 2; p.batch = batch; p.sliced = sliced;
    p.spc = sliced ? batch : 0;
    p.bands.clear();
    return NSGCQT_OK;
}

int finish_plan(HostPlan& p, std::string& err);

}  // namespace

int build_host_plan(HostPlan& p, double fs, double fmin, double fmax, int B,
                    int64_t N, int batch, bool sliced, std::string& err) {
    if (int r = begin_plan(p, fs, N, batch, sliced, err)) return r;
    if (!(fmin > 0.0) || !(fmin < fs / 2.0))
        return fail(err, NSGCQT_EINVAL, "fmin must satisfy 0 < fmin < fs/2");
    if (!(fmax >= fmin)) return fail(err, NSGCQT_EINVAL, "fmax must be >= fmin");
    if (B < 1) return fail(err, NSGCQT_EINVAL, "bins_per_octave must be >= 1");
    p.fmin = fmin; p.fmax = fmax; p.bpo = B;
    const int64_t half = N / 2;

    // ---- layout: geometric centres, Hann windows, DC and Nyquist sidebands
    const double Q = 1.0 / (std::pow(2.0, 1.0 / B) - 1.0);
    std::vector<double> fc, xis, betas;
    for (int j = 0;; ++j) {
        const double f = fmin * std::pow(2.0, static_cast<double>(j) / B);
        if (!(f <= fmax * (1.0 + 1e-12) && f < fs / 2.0)) break;
        fc.push_back(f);
        xis.push_back(f * static_cast<double>(N) / fs);
        betas.push_back((f / Q) * static_cast<double>(N) / fs);
    }
    {
        const double xi0 = xis.front(), b0 = betas.front();
        HostBand b{};
        b.kind = 0; b.k_lo = 0; b.k_hi = static_cast<int64_t>(std::ceil(xi0)) - 1; b.k_c = 0;
        b.f = 0.0; b.xi = xi0; b.beta = b0;
        for (int64_t k = b.k_lo; k <= b.k_hi; ++k) {
            const double kd = static_cast<double>(k);
            const double s = std::sin(kPi * (xi0 - kd) / (2.0 * b0));
            b.g.push_back(kd <= xi0 - b0 ? 1.0 : s * s);
        }
        p.bands.push_back(std::move(b));
    }
    for (size_t j = 0; j < fc.size(); ++j) {
        const double xi = xis[j], beta = betas[j];
        const int64_t k_lo = std::max<int64_t>(0, static_cast<int64_t>(std::floor(xi - beta)) + 1);
        const int64_t k_hi = std::min<int64_t>(half, static_cast<int64_t>(std::ceil(xi + beta)) - 1);
        if (k_hi < k_lo) continue;
        HostBand b{};
        b.kind = 1; b.k_lo = k_lo; b.k_hi = k_hi;
        b.k_c = static_cast<int64_t>(std::floor(xi + 0.5));
        b.f = fc[j]; b.xi = xi; b.beta = beta;
        for (int64_t k = k_lo; k <= k_hi; ++k) {
            const double c = std::cos(kPi * (static_cast<double>(k) - xi) / (2.0 * beta));
            b.g.push_back(c * c);
        }
        p.bands.push_back(std::move(b));
    }
    {
        const double xl = xis.back(), bl = betas.back();
        HostBand b{};
        b.kind = 2; b.k_lo = static_cast<int64_t>(std::floor(xl)) + 1; b.k_hi = half; b.k_c = half;
        b.f = fs / 2.0; b.xi = xl; b.beta = bl;
        for (int64_t k = b.k_lo; k <= b.k_hi; ++k) {
            const double kd = static_cast<double>(k);
            const double s = std::sin(kPi * (kd - xl) / (2.0 * bl));
            b.g.push_back(kd >= xl + bl ? 1.0 : s * s);
        }
        p.bands.push_back(std::move(b));
    }
    // constant-Q bands are as long as their support
    for (auto& b : p.bands) b.M = b.width();
    return finish_plan(p, err);
}

int build_host_plan_bands(HostPlan& p, double fs, int64_t N, int batch, const std::vector<BandSpec>& specs,
                          bool sliced, std::string& err) {
    if (int r = begin_plan(p, fs, N, batch, sliced, err)) return r;
    p.fmin = 0.0; p.fmax = 0.0; p.bpo = 0;
    if (specs.empty()) return fail(err, NSGCQT_EINVAL, "the band list is empty");
    if (specs.size() >= (size_t(1) << 24)) return fail(err, NSGCQT_EUNSUPPORTED, "too many bands");
    const int64_t half = N / 2;
    for (size_t i = 0; i < specs.size(); ++i) {
        const BandSpec& s = specs[i];
        const std::string name = "band " + std::to_string(i);
        if (s.kind < 0 || s.kind > 2) return fail(err, NSGCQT_EINVAL, name + ": kind must be 0, 1 or 2");
        if (s.kind == 0 && i != 0) return fail(err, NSGCQT_EINVAL, name + ": a DC band must come first");
        if (s.kind == 2 && i + 1 != specs.size()) return fail(err, NSGCQT_EINVAL, name + ": a Nyquist band must come last");
        if (!std::isfinite(s.xi) || !(s.beta > 0.0) || !std::isfinite(s.beta) || std::fabs(s.xi) > 1e15 || s.beta > 1e15)
            return fail(err, NSGCQT_EINVAL, name + ": xi must be finite and beta finite and > 0");
        if (s.M < 0) return fail(err, NSGCQT_EINVAL, name + ": length must be >= 0");
        HostBand b{};
        b.kind = s.kind; b.xi = s.xi; b.beta = s.beta; b.f = s.f;
        if (s.kind == 0) {
            // flat, then a sin^2 taper complementing the lower half of the Hann window at xi
            b.k_lo = 0;
            b.k_hi = std::min<int64_t>(half, static_cast<int64_t>(std::ceil(s.xi)) - 1);
            b.k_c = 0;
            for (int64_t k = b.k_lo; k <= b.k_hi; ++k) {
                const double kd = static_cast<double>(k);
                const double sn = std::sin(kPi * (s.xi - kd) / (2.0 * s.beta));
                b.g.push_back(kd <= s.xi - s.beta ? 1.0 : sn * sn);
            }
        } else if (s.kind == 1) {
            b.k_lo = std::max<int64_t>(0, static_cast<int64_t>(std::floor(s.xi - s.beta)) + 1);
            b.k_hi = std::min<int64_t>(half, static_cast<int64_t>(std::ceil(s.xi + s.beta)) - 1);
            b.k_c = static_cast<int64_t>(std::floor(s.xi + 0.5));
            for (int64_t k = b.k_lo; k <= b.k_hi; ++k) {
                const double c = std::cos(kPi * (static_cast<double>(k) - s.xi) / (2.0 * s.beta));
                b.g.push_back(c * c);
            }
        } else {
            // a sin^2 taper complementing the upper half of the Hann window at xi, then flat
            b.k_lo = std::max<int64_t>(0, static_cast<int64_t>(std::floor(s.xi)) + 1);
            b.k_hi = half;
            b.k_c = half;
            for (int64_t k = b.k_lo; k <= b.k_hi; ++k) {
                const double kd = static_cast<double>(k);
                const double sn = std::sin(kPi * (kd - s.xi) / (2.0 * s.beta));
                b.g.push_back(kd >= s.xi + s.beta ? 1.0 : sn * sn);
            }
        }
        if (b.k_hi < b.k_lo) return fail(err, NSGCQT_EINVAL, name + ": empty support");
        b.M = s.M ? s.M : b.width();
        if (b.M < b.width())
            return fail(err, NSGCQT_EINVAL, name + ": length " + std::to_string(b.M) + " below its support width " +
                                                std::to_string(b.width()));
        if (b.M >= (int64_t(1) << 28)) return fail(err, NSGCQT_EUNSUPPORTED, name + ": length of 2^28 or more");
        p.bands.push_back(std::move(b));
    }
    return finish_plan(p, err);
}

void table1_specs(std::vector<BandSpec>& out) {
    // Nine octaves above a lowest centre of 64 bins (43.07 Hz): octaves 1-3
    // at 8, 4-7 at 16 and 8-9 at 32 bands per octave. Centre j of octave o
    // is 64 * 2^(o + j/B) bins (o from 0), rounded to a bin; the highest
    // centre is the table's 21,810 Hz, rounded to a bin. Each Hann window
    // has half-amplitude width xi/Q with Q = 1/(2^(1/B) - 1) of its octave.
    // Every band of an octave has the length of the octave's widest
    // support, rounded up to a power of two; the DC and Nyquist sidebands
    // have lengths 128 and 2048.
    static const int kBpo[9] = {8, 8, 8, 16, 16, 16, 16, 32, 32};
    const double N = static_cast<double>(kTable1N), fs = kTable1Fs;
    const int64_t half = kTable1N / 2;
    out.clear();
    std::vector<BandSpec> pos;
    std::vector<int> oct;
    for (int o = 0; o < 9; ++o) {
        const int B = kBpo[o];
        for (int j = 0; j < B; ++j) {
            BandSpec s{};
            s.kind = 1;
            s.xi = std::nearbyint(64.0 * std::pow(2.0, o + static_cast<double>(j) / B));
            pos.push_back(s);
            oct.push_back(o);
        }
    }
    pos.back().xi = std::nearbyint(21810.0 * N / fs);
    for (size_t i = 0; i < pos.size(); ++i) {
        const double Q = 1.0 / (std::pow(2.0, 1.0 / kBpo[oct[i]]) - 1.0);
        pos[i].beta = pos[i].xi / Q;
        pos[i].f = pos[i].xi * fs / N;
    }
    int64_t widest[9] = {0};
    for (size_t i = 0; i < pos.size(); ++i) {
        const int64_t lo = std::max<int64_t>(0, static_cast<int64_t>(std::floor(pos[i].xi - pos[i].beta)) + 1);
        const int64_t hi = std::min<int64_t>(half, static_cast<int64_t>(std::ceil(pos[i].xi + pos[i].beta)) - 1);
        widest[oct[i]] = std::max(widest[oct[i]], hi - lo + 1);
    }
    for (size_t i = 0; i < pos.size(); ++i) {
        int64_t M = 1;
        while (M < widest[oct[i]]) M *= 2;
        pos[i].M = M;
    }
    out.push_back(BandSpec{0, pos.front().xi, pos.front().beta, 128, 0.0});
    out.insert(out.end(), pos.begin(), pos.end());
    out.push_back(BandSpec{2, pos.back().xi, pos.back().beta, 2048, fs / 2.0});
}

int erb_specs(double fs, int64_t N, double fmin, double fmax, double v, std::vector<BandSpec>& out,
              std::string& err) {
    out.clear();
    if (!(N >= 4) || (N % 2) != 0) return fail(err, NSGCQT_EINVAL, "n_samples must be even and >= 4");
    if (!(fs > 0.0)) return fail(err, NSGCQT_EINVAL, "fs must be > 0");
    if (!(fmin > 0.0) || !(fmin < fs / 2.0)) return fail(err, NSGCQT_EINVAL, "fmin must satisfy 0 < fmin < fs/2");
    if (!(fmax >= fmin)) return fail(err, NSGCQT_EINVAL, "fmax must be >= fmin");
    if (!(v > 0.0) || !(v <= 1e3)) return fail(err, NSGCQT_EINVAL, "bands per ERB must be in (0, 1000]");
    // Glasberg and Moore: ERB(f) = 24.7 (4.37 f / 1000 + 1) Hz and the
    // ERB-rate E(f) = 21.4 log10(1 + 4.37 f / 1000)
    auto erb = [](double f) { return 24.7 * (4.37 * f / 1000.0 + 1.0); };
    auto rate = [](double f) { return 21.4 * std::log10(1.0 + 4.37 * f / 1000.0); };
    auto inv_rate = [](double e) { return (std::pow(10.0, e / 21.4) - 1.0) * 1000.0 / 4.37; };
    const double Nd = static_cast<double>(N), e0 = rate(fmin);
    const int64_t half = N / 2;
    std::vector<BandSpec> pos;
    for (int64_t j = 0;; ++j) {
        const double f = inv_rate(e0 + static_cast<double>(j) / v);
        if (!(f <= fmax * (1.0 + 1e-12) && f < fs / 2.0)) break;
        if (j > 1000000) return fail(err, NSGCQT_EUNSUPPORTED, "more than a million bands");
        BandSpec s{};
        s.kind = 1;
        s.xi = f * Nd / fs;
        s.beta = erb(f) / v * Nd / fs;
        s.M = 0;
        s.f = f;
        const int64_t lo = std::max<int64_t>(0, static_cast<int64_t>(std::floor(s.xi - s.beta)) + 1);
        const int64_t hi = std::min<int64_t>(half, static_cast<int64_t>(std::ceil(s.xi + s.beta)) - 1);
        if (hi >= lo) pos.push_back(s);
    }
    if (pos.empty()) return fail(err, NSGCQT_EINVAL, "no band between fmin and fmax");
    out.push_back(BandSpec{0, pos.front().xi, pos.front().beta, 0, 0.0});
    out.insert(out.end(), pos.begin(), pos.end());
    out.push_back(BandSpec{2, pos.back().xi, pos.back().beta, 0, fs / 2.0});
    return NSGCQT_OK;
}

namespace {

int finish_plan(HostPlan& p, std::string& err) {
    const int64_t N = p.N, L = p.L, half = N / 2;
    const int batch = p.batch;
    const bool sliced = p.sliced;

    // ---- aggregate weight and dual windows (Sec. 2)
    p.a.assign(half + 1, 0.0);
    int64_t off = 0;
    p.maxM = 0;
    for (auto& b : p.bands) {
        b.off = off;
        off += b.M;
        p.maxM = std::max(p.maxM, b.M);
        for (int64_t i = 0; i < b.width(); ++i) p.a[b.k_lo + i] += static_cast<double>(b.M) * b.g[i] * b.g[i];
    }
    p.C = off;
    for (int64_t k = 0; k <= half; ++k)
        if (!(p.a[k] > 0.0)) return fail(err, NSGCQT_EINVAL, "layout leaves bin " + std::to_string(k) + " uncovered (a_k = 0)");
    if (p.C * static_cast<int64_t>(batch) * 8 > (int64_t(1) << 46))
        return fail(err, NSGCQT_EUNSUPPORTED, "coefficient array too large");
    for (auto& b : p.bands) {
        b.h.resize(b.width());
        for (int64_t i = 0; i < b.width(); ++i) b.h[i] = static_cast<double>(b.M) * b.g[i] / p.a[b.k_lo + i];
    }

    // ---- per-coefficient weight tables in bin order (Sec. 3, eq. 7 and Sec. 3.2);
    // the entries of a band past its support are zero
    p.wA.assign(p.C, 0.f); p.wS.assign(p.C, 0.f); p.wT.assign(p.C, 0.f); p.wSa.assign(p.C, 0.f);
    for (auto& b : p.bands)
        for (int64_t i = 0; i < b.width(); ++i) {
            const int64_t k = b.k_lo + i;
            const double d = (k == 0 || k == half) ? 1.0 : 2.0;
            const double M = static_cast<double>(b.M);
            p.wA[b.off + i] = static_cast<float>(b.g[i]);
            p.wS[b.off + i] = static_cast<float>(b.h[i]);
            p.wT[b.off + i] = static_cast<float>(static_cast<double>(N) / (d * M) * b.g[i]);
            p.wSa[b.off + i] = static_cast<float>(M * d / static_cast<double>(N) * b.h[i]);
        }
    // router factors (eq. 7) in fp64, rounded once
    p.rA.assign(4 * p.C, 0.f); p.rSa.assign(4 * p.C, 0.f);
    for (auto& b : p.bands)
        for (int64_t i = 0; i < b.width(); ++i) {
            const int64_t k = b.k_lo + i;
            const double d = (k == 0 || k == half) ? 1.0 : 2.0;
            const cd w = root(k, N), iw = cd(0.0, 1.0) * w;
            const double wts[2] = {b.g[i], static_cast<double>(b.M) * d / static_cast<double>(N) * b.h[i]};
            std::vector<float>* dst[2] = {&p.rA, &p.rSa};
            for (int t = 0; t < 2; ++t) {
                const cd pa = 0.5 * wts[t] * (1.0 - iw), pb = 0.5 * wts[t] * (1.0 + iw);
                float* o = dst[t]->data() + 4 * (b.off + i);
                o[0] = static_cast<float>(pa.real());
                o[1] = static_cast<float>(pa.imag());
                o[2] = static_cast<float>(pb.real());
                o[3] = static_cast<float>(pb.imag());
            }
        }

    // ---- bin ownership for the overlap-add and fan-out statistics
    p.owner.assign(half + 1, -1);
    std::vector<int32_t> cnt(half + 1, 0);
    for (size_t l = 0; l < p.bands.size(); ++l) {
        const auto& b = p.bands[l];
        for (int64_t k = b.k_lo; k <= b.k_hi; ++k) {
            if (p.owner[k] < 0) p.owner[k] = static_cast<int32_t>(l);
            else if (p.owner[k] + cnt[k] != static_cast<int32_t>(l))
                return fail(err, NSGCQT_EUNSUPPORTED, "bands covering a bin are not consecutive");
            ++cnt[k];
        }
    }
    p.max_overlap = 0;
    for (int64_t k = 0; k <= half; ++k) {
        if (cnt[k] > 127 || p.bands.size() >= (1u << 24))
            return fail(err, NSGCQT_EUNSUPPORTED, "too many bands per bin");
        p.max_overlap = std::max<int64_t>(p.max_overlap, cnt[k]);
        p.owner[k] |= cnt[k] << 24;
    }
    {
        std::vector<int32_t> fan(L / 2 + 1, 0);
        for (const auto& b : p.bands)
            for (int64_t k = b.k_lo; k <= b.k_hi; ++k) {
                const int64_t q = k % L, r = (L - q) % L;
                ++fan[std::min(q, r)];
            }
        p.max_fanout = *std::max_element(fan.begin(), fan.end());
    }
    p.bandbase.resize(p.bands.size());
    for (size_t l = 0; l < p.bands.size(); ++l)
        p.bandbase[l] = static_cast<int32_t>(p.bands[l].off - p.bands[l].k_lo);
    // per bin k, one record for the bin and its mirror L - k, so the
    // overlap-add reads both with one table load. For each side: the W index
    // (within one signal's row) of the first covering band with the count in
    // its top 3 bits, then the second and third bands' W indices. Compact
    // (16 bytes): those two as int16 steps from the previous index (0 where
    // there is no such band). Wide (32 bytes, when a step does not fit 16
    // bits): absolute indices, the first band's where there is no such band;
    // layout head_k, i1_k, i2_k, head_m | i1_m, i2_m, 0, 0.
    if (p.max_overlap > 3) return fail(err, NSGCQT_EUNSUPPORTED, "more than three bands cover one bin");
    if (p.C >= (int64_t(1) << 29)) return fail(err, NSGCQT_EUNSUPPORTED, "2^29 coefficients or more");
    {
        std::vector<int32_t> head(half + 1), i1(half + 1), i2(half + 1), steps(half + 1);
        bool wide = false;
        for (int64_t k = 0; k <= half; ++k) {
            const int first = p.owner[k] & 0xFFFFFF, cnt = p.owner[k] >> 24;
            int64_t idx[3] = {0, 0, 0};
            for (int j = 0; j < cnt; ++j) idx[j] = p.bandbase[first + j] + k;
            const int64_t d1 = cnt > 1 ? idx[1] - idx[0] : 0, d2 = cnt > 2 ? idx[2] - idx[1] : 0;
            if (d1 < -32768 || d1 > 32767 || d2 < -32768 || d2 > 32767) wide = true;
            head[k] = static_cast<int32_t>(idx[0] | (static_cast<int64_t>(cnt) << 29));
            i1[k] = static_cast<int32_t>(cnt > 1 ? idx[1] : idx[0]);
            i2[k] = static_cast<int32_t>(cnt > 2 ? idx[2] : idx[0]);
            steps[k] = static_cast<int32_t>((d1 & 0xFFFF) | (static_cast<uint32_t>(d2 & 0xFFFF) << 16));
        }
        p.gather_wide = wide;
        p.gather.assign((wide ? 8 : 4) * (half + 1), 0);
        for (int64_t k = 0; k <= half; ++k) {
            const int64_t m = L - k;   // mirror bin (0 <-> L)
            if (wide) {
                int32_t* r = p.gather.data() + 8 * k;
                r[0] = head[k]; r[1] = i1[k]; r[2] = i2[k]; r[3] = head[m];
                r[4] = i1[m]; r[5] = i2[m];
            } else {
                int32_t* r = p.gather.data() + 4 * k;
                r[0] = head[k]; r[1] = steps[k]; r[2] = head[m]; r[3] = steps[m];
            }
        }
    }

    // ---- omega_k = exp(-2 pi i k / N) for the untangle (eq. 6) and retangle (eq. 9)
    p.omega.clear();
    for (int64_t k = 0; k <= L; ++k) push_c(p.omega, root(k, N));

    // ---- packed FFT: four-step split L = L1 * L2
    p.ffts.clear(); p.twpool.clear();
    FftRegistry reg(p);
    {
        int64_t best = -1;
        for (int64_t d = 1; d * d <= L; ++d) {
            if (L % d) continue;
            std::vector<int> r1, r2;
            if (factor_radices(d, r1) && factor_radices(L / d, r2)) best = d;
        }
        if (best < 0)
            return fail(err, NSGCQT_EUNSUPPORTED,
                        "packed length L = " + std::to_string(L) + " has a prime factor above " +
                            std::to_string(kMfmaMaxRadix));
        auto& f = p.fs4;
        f.L1 = best; f.L2 = L / best;
        if (f.L2 > 8192) return fail(err, NSGCQT_EUNSUPPORTED, "packed length too large for the two-pass FFT");
        f.fft1 = reg.get(f.L1);
        f.fft2 = reg.get(f.L2);
        // up to 16 sequences per workgroup (a power of two), at most 8
        // elements per thread; fewer (down to 2) while the pass would have
        // fewer than kPassTiles tiles, so that small batches still spread
        // over the device (each sequence's arithmetic does not depend on
        // how many share a workgroup)
        const int64_t nsig = batch;
        auto pick = [nsig](int64_t n, int64_t count, int& lgt, int& nt) {
            lgt = 4;
            while (lgt > 0 && ((int64_t(1) << lgt) * n > 8192 || (int64_t(1) << (lgt - 1)) >= count)) --lgt;
            while (lgt > 1 && ((count + (int64_t(1) << lgt) - 1) >> lgt) * nsig < kPassTiles) --lgt;
            nt = 1024;
            for (int t : {256, 512, 1024})
                if ((int64_t(1) << lgt) * n <= 8 * t) { nt = t; break; }
        };
        pick(f.L1, f.L2, f.tile_a, f.nt_a);
        pick(f.L2, f.L1, f.tile_b, f.nt_b);
        // the sliced pass A also carries the two samples' clamped positions
        // and window values per element: at most 512 threads x 8 elements,
        // so its registers fit without spilling
        if (sliced) {
            if (f.L1 > 4096)
                return fail(err, NSGCQT_EUNSUPPORTED, "slice length too large for the sliced column pass");
            while (f.tile_a > 0 && (int64_t(1) << f.tile_a) * f.L1 > 4096) --f.tile_a;
            f.nt_a = std::min(f.nt_a, 512);
        }
        if ((int64_t(1) << f.tile_a) * f.L1 > 8192 || (int64_t(1) << f.tile_b) * f.L2 > 8192)
            return fail(err, NSGCQT_EUNSUPPORTED, "four-step pass exceeds one workgroup");
        // fewer columns per workgroup until the prime stages' matrix tiles fit
        {
            std::vector<int> r1, r2;
            factor_radices(f.L1, r1);
            factor_radices(f.L2, r2);
            while (f.tile_a > 0 && !mfma_fits(r1, f.L1, f.tile_a, f.nt_a)) --f.tile_a;
            while (f.tile_b > 0 && !mfma_fits(r2, f.L2, f.tile_b, f.nt_b)) --f.tile_b;
            if (!mfma_fits(r1, f.L1, f.tile_a, f.nt_a) || !mfma_fits(r2, f.L2, f.tile_b, f.nt_b))
                return fail(err, NSGCQT_EUNSUPPORTED, "four-step pass: prime stage exceeds the workgroup");
        }
        {
            int lg4 = 0;
            while ((int64_t(1) << (2 * lg4)) < L) ++lg4;
            const int64_t t4 = ((L + (int64_t(1) << lg4) - 1) >> lg4) + (int64_t(1) << lg4);
            const int64_t a_slots = t4 + p.ffts[f.fft1].ntw + lds_slots(static_cast<int>(f.L1), f.tile_a);
            const int64_t b_slots = p.ffts[f.fft2].ntw + lds_slots(static_cast<int>(f.L2), f.tile_b);
            if (a_slots * 8 > 160 * 1024 || b_slots * 8 > 160 * 1024)
                return fail(err, NSGCQT_EUNSUPPORTED, "four-step pass exceeds LDS");
        }
        int lg = 0;
        while ((int64_t(1) << (2 * lg)) < L) ++lg;
        const int64_t s = int64_t(1) << lg;
        f.split = lg;
        p.tw4_hi.clear(); p.tw4_lo.clear();
        for (int64_t i = 0; i * s < L; ++i) push_c(p.tw4_hi, root(i * s, L));
        for (int64_t j = 0; j < s; ++j) push_c(p.tw4_lo, root(j, L));
    }

    // ---- band transforms: mixed radix, or Bluestein over a smooth length
    p.banddev.clear(); p.chirp.clear(); p.kern.clear();
    const int64_t row_bytes = std::max<int64_t>(p.L + 1, p.C) * 8;
    std::vector<int> work(p.bands.size());
    std::vector<BandFit> fit(p.bands.size());
    for (size_t l = 0; l < p.bands.size(); ++l) {
        const auto& b = p.bands[l];
        BandDev d{};
        d.k_lo = static_cast<int32_t>(b.k_lo);
        d.M = static_cast<int32_t>(b.M);
        d.W = static_cast<int32_t>(b.width());
        d.rot = static_cast<int32_t>(((b.k_lo - b.k_c) % b.M + b.M) % b.M);
        d.off = static_cast<int32_t>(b.off);
        d.inv_M = static_cast<float>(1.0 / static_cast<double>(b.M));
        d.chirp = -1; d.kern = -1;
        // direct transform of length M, or Bluestein over P, whichever the
        // cost model prefers
        const int64_t M = b.M;
        double c_blu = 0.0;
        const int64_t P = bluestein_length(M, row_bytes, &c_blu);
        const BandFit fd = band_fft_fit(M, row_bytes);
        if (fd.cost <= c_blu || P < 0) {
            fit[l] = fd;
            d.fft = reg.get(M);
            if (d.fft < 0) return fail(err, NSGCQT_EUNSUPPORTED, "no radix plan for a band");
            work[l] = static_cast<int>(M);
            d.n = static_cast<int32_t>(M);
        } else {
            d.fft = reg.get(P);
            if (d.fft < 0) return fail(err, NSGCQT_EUNSUPPORTED, "no Bluestein length");
            d.chirp = static_cast<int32_t>(p.chirp.size() / 2);
            d.kern = static_cast<int32_t>(p.kern.size() / 2);
            // chirp exp(-i pi m^2 / M), argument reduced exactly: m^2 mod 2M
            std::vector<cd> ch(M);
            for (int64_t m = 0; m < M; ++m) {
                const int64_t t = (m * m) % (2 * M);
                const double ang = kPi * static_cast<double>(t) / static_cast<double>(M);
                ch[m] = cd(std::cos(ang), -std::sin(ang));
                push_c(p.chirp, ch[m]);
            }
            // kernel b_P[t] = conj(chirp[|t|]) on the cyclic support |t| < M,
            // transformed once and scaled by 1/P
            std::vector<cd> bp(P, cd(0.0, 0.0));
            for (int64_t t = 0; t < M; ++t) {
                bp[t] = std::conj(ch[t]);
                if (t) bp[P - t] = std::conj(ch[t]);
            }
            host_dft(bp);
            for (int64_t t = 0; t < P; ++t) push_c(p.kern, bp[t] / static_cast<double>(P));
            work[l] = static_cast<int>(P);
            d.n = static_cast<int32_t>(P);
            fit[l] = band_fft_fit(P, row_bytes);
        }
        p.banddev.push_back(d);
    }

    // ---- buckets by transform length
    p.buckets.clear();
    for (const auto& t : kTiers) {
        Bucket bk{};
        bk.nt = t.nt; bk.ept = t.ept; bk.max_work = 0; bk.coeffs = 0;
        p.buckets.push_back(bk);
    }
    p.bigs.clear(); p.bigitems.clear(); p.Hn = 0; p.C_big = 0; p.Hn_blu = 0; p.C_big_blu = 0;
    int big_t4 = 0, big_ea = 0, big_eb = 0;
    for (size_t l = 0; l < p.bands.size(); ++l) {
        const int ti = fit[l].tier;
        if (ti < 0) {
            // four-step through global memory: n = n1 n2, n1 <= n2 <= 4096
            const int64_t n = work[l];
            const int64_t n1 = huge_split(n);
            if (n1 < 0)
                return fail(err, NSGCQT_EUNSUPPORTED,
                            "band of length " + std::to_string(p.bands[l].M) + " needs a transform of " +
                                std::to_string(n) + " points with no supported four-step split");
            BigDesc g{};
            g.band = static_cast<int32_t>(l);
            g.n = static_cast<int32_t>(n);
            g.n1 = static_cast<int32_t>(n1);
            g.n2 = static_cast<int32_t>(n / n1);
            g.fftn = reg.get(n);
            g.fft1 = reg.get(g.n1);
            g.fft2 = reg.get(g.n2);
            if (g.fftn < 0 || g.fft1 < 0 || g.fft2 < 0)
                return fail(err, NSGCQT_EUNSUPPORTED, "huge band transform has no radix plan");
            // columns / rows per workgroup of 512 threads: at most 16, within
            // 4096 elements, and with the prime stages' matrix tiles fitting
            std::vector<int> r1, r2;
            factor_radices(g.n1, r1);
            factor_radices(g.n2, r2);
            g.lga = 4;
            while (g.lga > 0 && ((1 << g.lga) * g.n1 > 4096 || (1 << (g.lga - 1)) >= g.n2 ||
                                 !mfma_fits(r1, g.n1, g.lga, 512)))
                --g.lga;
            g.lgb = 4;
            while (g.lgb > 0 && ((1 << g.lgb) * g.n2 > 4096 || (1 << (g.lgb - 1)) >= g.n1 ||
                                 !mfma_fits(r2, g.n2, g.lgb, 512)))
                --g.lgb;
            if (!mfma_fits(r1, g.n1, g.lga, 512) || !mfma_fits(r2, g.n2, g.lgb, 512))
                return fail(err, NSGCQT_EUNSUPPORTED, "huge band: prime stage exceeds the workgroup");
            g.hoff = static_cast<int32_t>(p.Hn);
            p.Hn += n;
            p.C_big += p.bands[l].M;
            if (p.banddev[l].chirp >= 0) { p.Hn_blu += n; p.C_big_blu += p.bands[l].M; }
            const FftDesc& fn = p.ffts[g.fftn];
            big_t4 = std::max(big_t4, fn.nhi + (1 << fn.lg));
            big_ea = std::max(big_ea, lds_slots(g.n1, g.lga));
            big_eb = std::max(big_eb, lds_slots(g.n2, g.lgb));
            p.bigs.push_back(g);
            continue;
        }
        auto& bk = p.buckets[ti];
        bk.bands.push_back(static_cast<int32_t>(l));
        bk.max_work = std::max(bk.max_work, work[l]);
        bk.coeffs += p.bands[l].M;
    }
    p.buckets.erase(std::remove_if(p.buckets.begin(), p.buckets.end(),
                                   [](const Bucket& b) { return b.bands.empty(); }),
                    p.buckets.end());
    // one work item per (band, group of signals): small transforms of one band
    // for several signals share a workgroup, up to nt * ept elements
    p.items.clear();
    for (auto& bk : p.buckets) {
        bk.item_off = static_cast<int>(p.items.size());
        const int E = bk.nt * bk.ept;
        bk.lds_elems = 0;
        for (int32_t l : bk.bands) {
            const int n = work[l];
            // 2^lg interleaved signals (seq_lg, within the band's matrix-tile cap)
            const int lg = std::min(seq_lg(n, E, batch, row_bytes), fit[l].lg_cap);
            const int G = 1 << lg;
            bk.lds_elems = std::max(bk.lds_elems, lds_slots(n, lg));
            // fast load phases (WorkItem flags): every read up to entry
            // M - 1 + 3 st of the band stays in the data or the guards
            const auto& hb = p.bands[static_cast<size_t>(l)];
            const int64_t st = bk.nt >> lg, reach = hb.M - 1 + 3 * st;
            int32_t fast = 0;
            if (hb.k_lo >= 1 && hb.k_lo + hb.M <= L && hb.k_lo + reach < L + kFastGuard && 3 * st <= L &&
                hb.off + reach < p.C + kFastGuard)
                fast |= kItemFastRoute;
            if (hb.off + reach < p.C) fast |= kItemFastCoef;
            for (int s0 = 0; s0 < batch; s0 += G)
                p.items.push_back(
                    WorkItem{l, s0, std::min(G, batch - s0), lg, fast, p.banddev[static_cast<size_t>(l)]});
        }
        bk.nitems = static_cast<int>(p.items.size()) - bk.item_off;
        if (bk.lds_elems * 8 > 160 * 1024)
            return fail(err, NSGCQT_EUNSUPPORTED, "band kernel exceeds LDS");
    }

    // huge-band work items: pass 0/1 over every huge band, pass 2/3 over the
    // Bluestein ones (their second FFT)
    for (int pass = 0; pass < 4; ++pass) {
        p.big_off[pass] = static_cast<int>(p.bigitems.size());
        for (size_t gi = 0; gi < p.bigs.size(); ++gi) {
            const BigDesc& g = p.bigs[gi];
            if (pass >= 2 && p.banddev[g.band].chirp < 0) continue;
            const int tiles = (pass % 2 == 0) ? (g.n2 + (1 << g.lga) - 1) >> g.lga : (g.n1 + (1 << g.lgb) - 1) >> g.lgb;
            for (int sg = 0; sg < batch; ++sg)
                for (int t = 0; t < tiles; ++t) p.bigitems.push_back(BigItem{static_cast<int32_t>(gi), sg, t, 0});
        }
        p.big_n[pass] = static_cast<int>(p.bigitems.size()) - p.big_off[pass];
    }
    p.big_lds_a = static_cast<int>((big_t4 + big_ea) * 8);
    p.big_lds_b = static_cast<int>(big_eb * 8);
    if (!p.bigs.empty() && (p.big_lds_a > 160 * 1024 || p.big_lds_b > 160 * 1024))
        return fail(err, NSGCQT_EUNSUPPORTED, "huge-band pass exceeds LDS");

    // ---- slicing window (Sec. 4): zero, sin^2 rise, flat, cos^2 fall, zero
    p.slicewin.clear();
    if (sliced) {
        const int64_t e = N / 8;
        const double q = static_cast<double>(N) / 2.0;
        for (int64_t t = 0; t < N; ++t) {
            double w = 0.0;
            if (t >= e && t < 3 * e) { const double s = std::sin(kPi * static_cast<double>(t - e) / q); w = s * s; }
            else if (t >= 3 * e && t < 5 * e) w = 1.0;
            else if (t >= 5 * e && t < 7 * e) { const double c = std::cos(kPi * static_cast<double>(t - 5 * e) / q); w = c * c; }
            p.slicewin.push_back(static_cast<float>(w));
        }
    }

    // ---- workspace
    const int64_t b = batch;
    const int64_t hbytes = p.Hn ? 2 * align256(8 * p.Hn * b) : 0;
    // the packed spectrum is followed by a guard for the band kernels' fast
    // router reads (kFastGuard entries)
    p.off_h_an = align256(8 * L * b) + align256(8 * L * b + 8 * static_cast<int64_t>(kFastGuard));
    p.ws_an = p.off_h_an + hbytes;
    p.off_h_syn = align256(8 * p.C * b) + align256(8 * L * b);
    p.off_y_sliced = p.off_h_syn + hbytes;
    p.ws_syn = p.off_y_sliced;
    if (sliced) p.ws_syn += align256(4 * N * b) + 2 * align256(4 * (N / 2));
    return NSGCQT_OK;
}

}  // namespace

}  // namespace nsg
