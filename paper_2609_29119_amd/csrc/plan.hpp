// Host-side plan: layout, windows, duals and every table the kernels read,
// computed in fp64 and stored as fp32 (or int32) for upload.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "tables.hpp"

namespace nsg {

struct HostBand {
    int kind;             // 0 DC, 1 positive, 2 Nyquist
    int64_t k_lo, k_hi, k_c;
    int64_t M;            // band length (transform length), at least the support width
    int64_t off;
    double f, xi, beta;
    std::vector<double> g, h;   // on k_lo..k_hi
    int64_t width() const { return k_hi - k_lo + 1; }
};

// One band of an explicit layout: the window kind (0 DC, 1 positive,
// 2 Nyquist), the centre xi and half-amplitude width beta (in bins) of the
// band's Hann window (for a sideband, of the neighbouring Hann window whose
// outer half it complements), and the band length M (0: the support width).
// f is the centre in Hz, reported only.
struct BandSpec {
    int kind;
    double xi, beta;
    int64_t M;
    double f;
};

// Band kernels are launched per bucket; each bucket has one thread count and
// one bound on the elements each thread holds per Stockham stage.
struct Bucket {
    int nt;               // threads per workgroup
    int ept;              // elements per thread bound (template parameter)
    int max_work;         // largest transform length in the bucket
    int64_t coeffs;       // sum of M over its bands
    std::vector<int32_t> bands;
    int item_off;         // first work item of the bucket in HostPlan::items
    int nitems;
    int lds_elems;        // largest data LDS slots over its items
};

// Four-step split of the packed FFT: L = L1 * L2. Pass A transforms columns
// (length L1, 2^tile_a columns per workgroup), pass B rows (length L2,
// 2^tile_b rows per workgroup).
struct FourStep {
    int64_t L1, L2;
    int fft1, fft2;       // FftDesc indices
    int tile_a, tile_b;   // log2 of the sequences per workgroup
    int nt_a, nt_b;       // threads per workgroup of each pass
    int64_t split;        // omega_L^t = hi[t >> split] * lo[t & (2^split - 1)]
};

struct HostPlan {
    // parameters
    double fs = 0, fmin = 0, fmax = 0;
    int bpo = 0;
    int64_t N = 0, L = 0;
    int batch = 0;
    bool sliced = false;
    int spc = 0;          // slices per chunk (sliced plans)

    // layout
    std::vector<HostBand> bands;
    int64_t C = 0, maxM = 0;
    int64_t max_fanout = 0, max_overlap = 0;
    std::vector<double> a;

    // fp32 tables
    std::vector<float> wA, wS, wT, wSa;     // C each, bin order
    // router factors of the analysis chains (T with g, S^dagger with its
    // weight w): (1/2) w (1 - i w_k) and (1/2) w (1 + i w_k) per coefficient,
    // as 4 floats (re, im, re, im), bin order
    std::vector<float> rA, rSa;
    std::vector<FftDesc> ffts;
    std::vector<float> twpool;              // interleaved complex
    std::vector<float> omega;               // exp(-2 pi i k / N), k = 0..L
    std::vector<float> tw4_hi, tw4_lo;      // four-step twiddles
    std::vector<int32_t> owner;             // per bin k = 0..L: first band | count << 24
    std::vector<int32_t> gather;            // per bin k = 0..L: covering bands of k and of L - k (see plan.cpp)
    bool gather_wide = false;               // 32-byte records with absolute indices (see plan.cpp)
    std::vector<int32_t> bandbase;          // per band: off - k_lo
    std::vector<BandDev> banddev;
    std::vector<float> chirp, kern;         // Bluestein tables
    std::vector<float> slicewin;            // sliced plans: window of length N
    std::vector<Bucket> buckets;
    std::vector<WorkItem> items;

    // huge bands (transform above one workgroup): descriptors, work items of
    // the four passes (all bands: column, row; Bluestein only: column, row)
    std::vector<BigDesc> bigs;
    std::vector<BigItem> bigitems;
    int big_off[4] = {0, 0, 0, 0}, big_n[4] = {0, 0, 0, 0};
    int64_t Hn = 0;             // complex values per signal in each huge-band buffer
    int64_t C_big = 0;          // coefficients of huge bands
    int64_t Hn_blu = 0;         // part of Hn that belongs to Bluestein bands
    int64_t C_big_blu = 0;      // coefficients of huge Bluestein bands
    int big_lds_a = 0, big_lds_b = 0;   // LDS bytes of the column / row passes
    FourStep fs4{};

    int64_t ws_an = 0, ws_syn = 0;
    int64_t off_h_an = 0, off_h_syn = 0, off_y_sliced = 0;   // workspace offsets
};

// Returns 0 on success, or a negative nsgcqt status with `err` set.
int build_host_plan(HostPlan& p, double fs, double fmin, double fmax, int bpo,
                    int64_t N, int batch, bool sliced, std::string& err);

// Plan of an explicit band list (see BandSpec); same return convention.
// sliced: N is the slice length and batch the slices per chunk.
int build_host_plan_bands(HostPlan& p, double fs, int64_t N, int batch, const std::vector<BandSpec>& specs,
                          bool sliced, std::string& err);

// The multi-resolution layout of the paper's Table 1 (N = 65,536 at 44.1 kHz).
constexpr int64_t kTable1N = 65536;
constexpr double kTable1Fs = 44100.0;
void table1_specs(std::vector<BandSpec>& out);

// An auditory (ERB-rate) layout for N samples at fs: positive centres
// equally spaced by 1/v on the ERB-rate scale from fmin while <= fmax and
// below fs/2, Hann windows whose half-amplitude width is the centre spacing
// ERB(f)/v, sidebands as in the constant-Q layout, lengths = support widths.
// Bands with empty support are left out. Returns 0 or a negative status.
int erb_specs(double fs, int64_t N, double fmin, double fmax, double v, std::vector<BandSpec>& out,
              std::string& err);

// Radix factorisation used by the Stockham stages: primes above 16 (at most
// max_prime) become stages of their own, the remaining factors are packed
// greedily into radices of at most 16. False when n has a larger prime factor
// or needs more than kMaxStages stages.
bool factor_radices(int64_t n, std::vector<int>& radices, int max_prime = kMfmaMaxRadix);

}  // namespace nsg
