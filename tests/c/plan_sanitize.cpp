// The host planner (plan.cpp) under AddressSanitizer, UBSan and libstdc++
// bounds assertions, over the workloads, the test layouts and the rejected
// inputs of the test suite. Prints one summary line; any sanitizer report or
// unexpected status makes the run fail.
#include <cmath>
#include <cstdio>
#include <string>
#include <vector>
#include "plan.hpp"
using namespace nsg;

static int n_ok = 0, n_err = 0, n_bad = 0;
static void cq(double fs, double fmin, double fmax, int B, int64_t N, int batch, bool sliced, bool expect_ok) {
    HostPlan p; std::string err;
    int r = build_host_plan(p, fs, fmin, fmax, B, N, batch, sliced, err);
    if ((r == 0) != expect_ok) {
        printf("UNEXPECTED cq fs=%g N=%lld B=%d r=%d %s\n", fs, (long long)N, B, r, err.c_str());
        ++n_bad;
    }
    (r == 0 ? n_ok : n_err)++;
}
static void bl(double fs, int64_t N, int batch, const std::vector<BandSpec>& s, bool sliced, bool expect_ok) {
    HostPlan p; std::string err;
    int r = build_host_plan_bands(p, fs, N, batch, s, sliced, err);
    if ((r == 0) != expect_ok) {
        printf("UNEXPECTED bands N=%lld r=%d %s\n", (long long)N, r, err.c_str());
        ++n_bad;
    }
    (r == 0 ? n_ok : n_err)++;
}
static std::vector<BandSpec> padded(const std::vector<double>& xs, const std::vector<int64_t>& lens, int64_t dc, int64_t ny) {
    std::vector<BandSpec> s;
    s.push_back({0, xs[0], xs[0] * 0.35, dc, 0.0});
    for (size_t i = 0; i < xs.size(); ++i) s.push_back({1, xs[i], xs[i] * 0.35, lens[i], 0.0});
    s.push_back({2, xs.back(), xs.back() * 0.35, ny, 0.0});
    return s;
}
int main() {
    // workloads
    cq(22050, 110, 11025, 12, 16384, 1, false, true);
    cq(44100, 32.7, 22050, 48, 44100, 1, false, true);
    cq(44100, 40, 22050, 24, 220500, 16, false, true);
    cq(22050, 55, 11025, 36, 88200, 128, false, true);
    cq(48000, 20, 24000, 96, 2880000, 1, false, true);
    cq(48000, 20, 24000, 96, 131072, 16, true, true);
    // small test layouts
    cq(4, 0.5, 2, 1, 4, 2, false, true);
    cq(6, 0.7, 3, 1, 6, 2, false, true);
    cq(8, 1, 4, 1, 8, 1, false, true);
    cq(30, 1, 15, 2, 30, 3, false, true);
    cq(250, 4, 125, 4, 500, 2, false, true);
    cq(268, 4, 134, 4, 268, 2, false, true);
    cq(1028, 8, 514, 6, 1028, 3, false, true);
    cq(250, 4, 125, 3, 250, 1, false, true);
    cq(4620, 30, 2310, 12, 4620, 3, false, true);
    cq(8000, 50, 4000, 24, 6000, 5, false, true);
    cq(22050, 110, 11025, 12, 16384, 3, false, true);
    // coarse long layout (wide gather records)
    cq(44100, 20, 22050, 12, 1323000, 1, false, true);
    // errors
    cq(22050, 110, 11025, 12, 16383, 1, false, false);   // odd N
    cq(22050, 110, 11025, 12, 2, 1, false, false);       // N < 4
    cq(22050, 11025, 11025, 12, 16384, 1, false, false); // fmin at Nyquist
    cq(22050, 110, 50, 12, 16384, 1, false, false);      // fmax < fmin
    cq(22050, 110, 11025, 0, 16384, 1, false, false);    // B < 1
    cq(22050, 110, 11025, 12, 16384, 0, false, false);   // batch < 1
    cq(-1, 110, 11025, 12, 16384, 1, false, false);      // fs <= 0
    // band lists
    std::vector<double> xs12, xs14;
    for (int j = 0; j < 12; ++j) xs12.push_back(8.0 * std::pow(1.35, j));
    for (int j = 0; j < 14; ++j) xs14.push_back(10.0 * std::pow(1.4, j));
    bl(1200, 1200, 2, padded(xs12, {0, 8, 0, 20, 0, 31, 40, 0, 67, 0, 2 * 263, 160}, 16, 1500), false, true);
    bl(4000, 4000, 2, padded(xs14, {0, 0, 0, 0, 0, 0, 8200, 0, 0, 8209, 0, 0, 0, 0}, 0, 9000), false, true);
    bl(4000, 4000, 2, padded(xs14, {512, 513, 2048, 2050, 4096, 4100, 8192, 8200, 16384, 16400, 0, 0, 0, 0}, 0, 0), false, true);
    bl(4000, 4000, 2, padded(xs14, {3, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0}, 0, 0), false, false);  // length below width
    std::vector<BandSpec> t1;
    table1_specs(t1);
    bl(44100, 65536, 128, t1, false, true);
    bl(44100, 65536, 1, t1, false, true);
    bl(44100, 65536, 16, t1, true, true);
    std::vector<BandSpec> erb; std::string err;
    if (erb_specs(16000, 32000, 50, 8000, 2.0, erb, err) != 0) {
        printf("UNEXPECTED erb %s\n", err.c_str());
        ++n_bad;
    }
    bl(16000, 32000, 2, erb, false, true);
    // maximum huge transform: N = 2^24, a DC band zero-padded to 2^24
    {
        const int64_t N = 1 << 24;
        const double h = double(N / 4);
        std::vector<BandSpec> s = {{0, h, 2.0, N, 0.0}, {1, h, 2.0, 0, 0.0}, {2, h, 2.0, 0, 0.0}};
        bl(48000.0, N, 1, s, false, true);
    }
    printf("plans ok %d, rejected %d, unexpected %d\n", n_ok, n_err, n_bad);
    return n_bad ? 1 : 0;
}
