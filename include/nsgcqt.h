/*
 * nsgcqt.h - C ABI of an exactly invertible nonstationary-Gabor constant-Q
 * transform (CQT) for AMD Instinct MI355X (gfx950).
 *
 * The transform is the one of "Exact Factorisation and Fast Computation of
 * Invertible Constant-Q Transforms" (Franchino, Moliner, Valimaki):
 *
 *   analysis   c_lambda = F_M^{-1} E_lambda diag(g_lambda) F_N x        (Sec. 2, eqs. 2-3)
 *   synthesis  x = F_N^{-1} sum_lambda diag(h_lambda) E^T F_M c_lambda  (Sec. 2, eq. 4)
 *   adjoints   T^dagger and S^dagger under <u,v> = Re(u^H v)         (Sec. 3.2, eqs. 13-14)
 *
 * evaluated through the packed factorisation of Sec. 3 (eqs. 5-10): one
 * length-L = N/2 FFT of the signal packed as complex pairs, a router that
 * untangles, windows, conjugates and reorders each band's bins, and one
 * length-M_lambda inverse FFT per band at the band's own length; synthesis
 * runs the reverse chain with one shared length-L inverse FFT.
 *
 * Conventions
 *   - DFT: [F_n]_{kj} = exp(-2 pi i k j / n), F_n^{-1} = F_n^H / n (eq. 1).
 *   - N (n_samples) is the number of real samples per signal and must be
 *     even; L = N/2.
 *   - Signals are [batch][N] float32, contiguous.
 *   - Coefficients are [batch][C] complex float32 stored as interleaved
 *     (re, im) float pairs, C = sum_lambda M_lambda. Band lambda occupies
 *     [offset_lambda, offset_lambda + M_lambda) of each row, in natural time
 *     order n = 0..M-1 (the output order of F_M^{-1}). Band order: DC
 *     sideband, positive bands by ascending centre, Nyquist sideband.
 *   - The band layout is the constant-Q layout: centres fmin 2^(j/B) up to
 *     fmax and below fs/2, Q = 1/(2^(1/B) - 1), Hann windows of
 *     half-amplitude width f/Q on the bins strictly inside +-f/Q of the
 *     centre, DC and Nyquist sidebands that complement the outer Hann
 *     halves, M = support width, the centre bin in slot 0. Dual windows are
 *     h = M g / a with a_k = sum M g^2 (Sec. 2). Bands with empty support
 *     are dropped at plan time.
 *   - Plans may instead take an explicit band list (nsgcqt_plan_create_bands):
 *     the same window shapes at given centres and widths, with lengths M at
 *     least the support width. Slots of a band past its support hold zero
 *     in analysis and are ignored by synthesis, as zero-padding the band
 *     spectrum to M (Sec. 2: E_lambda places the support injectively).
 *
 * Pointers and ownership
 *   - x, coeffs, outputs and the workspace are device pointers owned by the
 *     caller. The workspace size comes from nsgcqt_plan_info(); the library
 *     never allocates during a compute call. Coefficients, the workspace and
 *     the signals of the non-sliced calls must be 8-byte aligned, the
 *     signals of the sliced calls 4-byte aligned (EINVAL otherwise).
 *   - A plan owns its device tables (allocated on the device current at
 *     creation, freed by nsgcqt_plan_destroy). Compute calls must be made
 *     with that device current; otherwise they return EINVAL and enqueue
 *     nothing. A plan's layout and tables are immutable. Calls on one plan from several host threads take turns
 *     while they enqueue (a per-plan lock); their work on different streams
 *     with distinct workspaces may then run concurrently on the device.
 *   - Compute calls only enqueue work (a hipStream_t, NULL for the default
 *     stream); they never synchronise the host and may be captured into a
 *     HIP graph. They are not in-place. When every band launch of a plan is
 *     small (few signals), independent launches of one call also run on the
 *     plan's own side streams, which wait for the work already on `stream`
 *     and which `stream` waits for before the call's later work: the call
 *     stays ordered on `stream` as one unit. Calls on one plan from several
 *     streams share those side streams and may partly serialise.
 *
 * Errors
 *   Every function returns an nsgcqt_status. No C++ exception crosses the
 *   ABI. The text of the last error on the calling thread is returned by
 *   nsgcqt_last_error(). EDEVICE reports only the HIP calls the library
 *   makes itself (each launch is checked by its own status): an error that
 *   an earlier HIP call of the caller left on the thread is neither
 *   reported nor cleared.
 */
#ifndef NSGCQT_H
#define NSGCQT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nsgcqt_plan_s* nsgcqt_plan;

typedef enum {
    NSGCQT_OK = 0,
    NSGCQT_EINVAL = -1,       /* invalid argument, null pointer, host-only plan */
    NSGCQT_ENOMEM = -2,       /* device or host allocation failed at plan time */
    NSGCQT_EDEVICE = -3,      /* a HIP call failed; see nsgcqt_last_error() */
    NSGCQT_EWORKSPACE = -4,   /* ws_bytes below the size the plan requires */
    NSGCQT_EUNSUPPORTED = -5  /* valid transform the library cannot evaluate */
} nsgcqt_status;

typedef enum {
    NSGCQT_OP_ANALYSE = 0,          /* T  : [b][N] f32 -> [b][C] c64 */
    NSGCQT_OP_SYNTHESISE = 1,       /* S  : [b][C] c64 -> [b][N] f32 */
    NSGCQT_OP_ADJ_ANALYSIS = 2,     /* T^dagger: [b][C] c64 -> [b][N] f32 */
    NSGCQT_OP_ADJ_SYNTHESIS = 3     /* S^dagger: [b][N] f32 -> [b][C] c64 */
} nsgcqt_op;

typedef enum { NSGCQT_BAND_DC = 0, NSGCQT_BAND_POSITIVE = 1, NSGCQT_BAND_NYQUIST = 2 } nsgcqt_band_kind;

typedef struct {
    int64_t kind;       /* nsgcqt_band_kind */
    int64_t k_lo;       /* first support bin */
    int64_t k_hi;       /* last support bin (inclusive) */
    int64_t k_centre;   /* bin placed in slot 0: slot(k) = (k - k_centre) mod M */
    int64_t length;     /* M >= k_hi - k_lo + 1 (equal for constant-Q plans) */
    int64_t offset;     /* first coefficient of the band in a row of C */
    double centre_hz;   /* 0 for DC, fs/2 for Nyquist */
    double xi;          /* centre in bins (unrounded) of the governing Hann window */
    double beta;        /* its half-amplitude width in bins */
    int64_t fft_len;    /* length of the band's DFT as evaluated: M for a direct
                           mixed-radix transform, P >= 2M - 1 for Bluestein */
    int64_t bluestein;  /* 1 if the band uses Bluestein's algorithm (two
                           length-P transforms), 0 otherwise; independent of batch */
} nsgcqt_band;

/* One band of an explicit layout (Sec. 2: window g, selection E, length M).
 * All widths and centres are in bins of the length-N DFT.
 *   NSGCQT_BAND_POSITIVE: Hann window g(k) = cos^2(pi (k - xi) / (2 beta)) on
 *       the bins with |k - xi| < beta, clipped to 0 <= k <= N/2; the bin
 *       floor(xi + 1/2) goes to slot 0.
 *   NSGCQT_BAND_DC: bins 0 <= k < xi, g = 1 for k <= xi - beta and
 *       sin^2(pi (xi - k) / (2 beta)) above (the complement of the lower half
 *       of a Hann window at xi, beta); bin 0 in slot 0. First band only.
 *   NSGCQT_BAND_NYQUIST: bins xi < k <= N/2, g = sin^2(pi (k - xi) / (2 beta))
 *       below xi + beta and 1 from there; bin N/2 in slot 0. Last band only.
 * slot(k) = (k - k_centre) mod length. length 0 means the support width. */
typedef struct {
    int32_t kind;       /* nsgcqt_band_kind */
    double xi;          /* centre in bins (sidebands: the neighbouring Hann's centre) */
    double beta;        /* half-amplitude width in bins, > 0 */
    int64_t length;     /* M >= support width, or 0 for the support width */
    double centre_hz;   /* reported by nsgcqt_band_info only */
} nsgcqt_band_spec;

typedef struct {
    int64_t n_bands;          /* bands kept */
    int64_t batch;            /* signals per call (slices per chunk for sliced plans) */
    int64_t n_samples;        /* N (slice length for sliced plans) */
    int64_t packed_len;       /* L = N/2 */
    int64_t total_coeffs;     /* C */
    int64_t max_band_len;     /* max M */
    int64_t max_fanout;       /* max over packed pairs {q, L-q} of band entries reading it (Sec. 3.1) */
    int64_t max_overlap;      /* max number of bands covering one bin */
    int64_t sliced;           /* 1 for a sliced plan */
    int64_t ws_analyse;       /* workspace bytes for nsgcqt_analyse / sliced analyse */
    int64_t ws_synthesise;    /* workspace bytes for nsgcqt_synthesise / sliced synthesise */
    int64_t ws_adjoint_analysis;   /* for NSGCQT_OP_ADJ_ANALYSIS */
    int64_t ws_adjoint_synthesis;  /* for NSGCQT_OP_ADJ_SYNTHESIS */
    int64_t table_bytes;      /* persistent device tables held by the plan */
    int64_t device_tables;    /* 1 if the plan holds device tables, 0 for host-only plans */
} nsgcqt_info;

/* Create a plan for `batch` signals of n_samples (= N, even, >= 4) real
 * samples at sample rate fs, with bands from fmin to fmax at bins_per_octave.
 * Builds every table in fp64 on the host and uploads fp32 copies to the
 * current HIP device.
 * EINVAL: out NULL, N odd or < 4, fs <= 0, fmin <= 0, fmin >= fs/2,
 *         fmax < fmin, bins_per_octave < 1, batch < 1, or a bin that no band
 *         covers (a_k = 0, Sec. 2).
 * EUNSUPPORTED: N >= 2^29 (rows are addressed with 32-bit byte offsets);
 *         L = N/2 has a prime factor above 257, the largest Stockham radix,
 *         or its two-pass split does not fit a workgroup's LDS (L above
 *         about 10^7; L = 2^23 fits);
 *         or a band transform beyond one workgroup has no split n = n1 n2
 *         with n1 <= n2 <= 4096 into such radices. Bands never need their
 *         length's prime factors to be small: Bluestein's algorithm covers
 *         any length. */
int nsgcqt_plan_create(nsgcqt_plan* out, double fs, double fmin, double fmax,
                       int bins_per_octave, int64_t n_samples, int batch);

/* Same layout and host tables as nsgcqt_plan_create, without touching any
 * device: for inspecting the layout and tables on machines without a GPU.
 * Compute calls on such a plan return EINVAL. */
int nsgcqt_plan_create_host(nsgcqt_plan* out, double fs, double fmin, double fmax,
                            int bins_per_octave, int64_t n_samples, int batch);

/* Sliced (streaming) plan, Sec. 4: slices of slice_len samples (a multiple
 * of 8) with 50 % overlap, a Tukey transition window that is 0 on the outer
 * eighths, sin^2 / cos^2 on the next quarters and 1 in the middle half, and
 * a front pad of slice_len/2 zeros. Slice s covers original samples
 * [s H - H, s H + H), H = slice_len/2, for s = 0 .. J-1, J = ceil(n/H) + 1.
 * Sliced calls process slices_per_chunk slices at a time, so the workspace
 * is bounded independently of the signal length. */
int nsgcqt_sliced_plan_create(nsgcqt_plan* out, double fs, double fmin, double fmax,
                              int bins_per_octave, int64_t slice_len, int slices_per_chunk);

/* Host-only variant of nsgcqt_sliced_plan_create. */
int nsgcqt_sliced_plan_create_host(nsgcqt_plan* out, double fs, double fmin, double fmax,
                                   int bins_per_octave, int64_t slice_len, int slices_per_chunk);

/* Plan of an explicit band list bands[0 .. n_bands-1] (nsgcqt_band_spec)
 * for `batch` signals of n_samples real samples at sample rate fs; the band
 * order is the coefficient order. Bands covering one bin must be adjacent in
 * the list (ascending centres satisfy this). Windows, dual windows and
 * every table follow exactly as for nsgcqt_plan_create.
 * EINVAL: out or bands NULL, n_bands < 1, N odd or < 4, fs <= 0, batch < 1,
 *         a kind other than 0..2, a DC band that is not first or a Nyquist
 *         band that is not last, xi not finite, beta not finite or <= 0,
 *         length < 0, a band with empty support, a length below the support
 *         width, or a bin no band covers (a_k = 0).
 * EUNSUPPORTED: as for nsgcqt_plan_create, and for bands covering one bin
 *         that are not adjacent, more than three bands on one bin, or a
 *         length of 2^28 or more. */
int nsgcqt_plan_create_bands(nsgcqt_plan* out, double fs, int64_t n_samples, int batch,
                             int n_bands, const nsgcqt_band_spec* bands);

/* Host-only variant of nsgcqt_plan_create_bands. */
int nsgcqt_plan_create_bands_host(nsgcqt_plan* out, double fs, int64_t n_samples, int batch,
                                  int n_bands, const nsgcqt_band_spec* bands);

/* Sliced (streaming) plan of an explicit band list for slices of slice_len
 * samples (a multiple of 8), with the slicing of nsgcqt_sliced_plan_create
 * (Sec. 4 streams the Table 1 layout this way). The bands are in bins of
 * the length-slice_len DFT. Errors as for nsgcqt_plan_create_bands, and
 * EINVAL for a slice length that is not a multiple of 8. */
int nsgcqt_sliced_plan_create_bands(nsgcqt_plan* out, double fs, int64_t slice_len, int slices_per_chunk,
                                    int n_bands, const nsgcqt_band_spec* bands);

/* Host-only variant of nsgcqt_sliced_plan_create_bands. */
int nsgcqt_sliced_plan_create_bands_host(nsgcqt_plan* out, double fs, int64_t slice_len,
                                         int slices_per_chunk, int n_bands, const nsgcqt_band_spec* bands);

/* The multi-resolution layout of Table 1 (Sec. 4): N = 65,536 at 44.1 kHz;
 * octaves 1-3 at 8, 4-7 at 16 and 8-9 at 32 bands per octave above a lowest
 * centre of 64 bins (43.07 Hz), centres rounded to bins and the highest one
 * at 21,810 Hz; each octave's bands share the length of its widest support
 * rounded up to a power of two; DC and Nyquist sidebands of lengths 128 and
 * 2048 (154 bands, C = 132,992). Writes the band count to *n_bands and, when
 * not NULL, the sample rate and length to *fs and *n_samples; with out
 * non-NULL also the bands, which need capacity >= *n_bands (EINVAL
 * otherwise). Pass the result to nsgcqt_plan_create_bands. */
int nsgcqt_layout_table1(nsgcqt_band_spec* out, int capacity, int* n_bands, double* fs,
                         int64_t* n_samples);

/* An auditory layout (another painless nonstationary Gabor frame, built like
 * the constant-Q one on the ERB-rate scale of Glasberg and Moore:
 * ERB(f) = 24.7 (4.37 f/1000 + 1) Hz, E(f) = 21.4 log10(1 + 4.37 f/1000)).
 * Positive centres f_j with E(f_j) = E(fmin) + j / bands_per_erb, kept while
 * f_j <= fmax and f_j < fs/2; Hann windows of half-amplitude width
 * ERB(f_j) / bands_per_erb (the centre spacing); DC and Nyquist sidebands
 * complementing the outer Hann halves; lengths = support widths; bands with
 * empty support left out. Fills *n_bands and, with out non-NULL, the bands
 * (capacity >= *n_bands, else EINVAL), for nsgcqt_plan_create_bands.
 * EINVAL: n_bands NULL, N odd or < 4, fs <= 0, fmin <= 0, fmin >= fs/2,
 *         fmax < fmin, bands_per_erb not in (0, 1000]. */
int nsgcqt_layout_erb(double fs, int64_t n_samples, double fmin, double fmax, double bands_per_erb,
                      nsgcqt_band_spec* out, int capacity, int* n_bands);

/* Free the plan and its device tables. Any work using it must have
 * completed. NULL is accepted. */
int nsgcqt_plan_destroy(nsgcqt_plan plan);

int nsgcqt_plan_info(nsgcqt_plan plan, nsgcqt_info* out);

/* Layout of band `band` (0 <= band < n_bands). EINVAL when out of range. */
int nsgcqt_band_info(nsgcqt_plan plan, int band, nsgcqt_band* out);

/* Host copies of the plan's per-coefficient fp32 weight tables, each C
 * floats in bin order (entry offset_lambda + (k - k_lo) belongs to bin k of
 * band lambda):
 *   0 g                                  analysis window
 *   1 h = M g / a                        synthesis dual window
 *   2 (N / (d_k M)) g                    weight of T^dagger
 *   3 (M d_k / N) h                      weight of S^dagger
 * with d_k = 1 at k = 0 and k = N/2 and 2 otherwise (Sec. 3.2).
 * `bytes` must be at least 4 C. */
int nsgcqt_plan_weights(nsgcqt_plan plan, int which, float* dst, size_t bytes);

/* T: x [batch][N] f32 -> coeffs [batch][C] c64 (eq. 8). */
int nsgcqt_analyse(nsgcqt_plan plan, const float* x, float* coeffs,
                   void* ws, size_t ws_bytes, void* stream);

/* Bytes of the device array that nsgcqt_analyse_noalloc uses as workspace. */
#define NSGCQT_NOALLOC_SCRATCH_BYTES (64u << 20)

/* T as nsgcqt_analyse, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels, with the workspace taken from a device
 * array of NSGCQT_NOALLOC_SCRATCH_BYTES that the library holds on every
 * device it runs on until the process ends. The call makes no allocation
 * of any kind. The caller still passes x and coeffs (as for
 * nsgcqt_analyse); nothing in the array needs to start at zero.
 * All calls on one device share that device's array, which keeps the last
 * call's contents: calls that overlap on one device (two streams, or two
 * host threads with unordered streams) race on it and give wrong results;
 * order them on one stream.
 * EWORKSPACE: the plan's analysis workspace (nsgcqt_info.ws_analyse)
 *             exceeds NSGCQT_NOALLOC_SCRATCH_BYTES.
 * EINVAL, EDEVICE: as nsgcqt_analyse (EDEVICE also when the array's device
 *             address cannot be obtained). */
int nsgcqt_analyse_noalloc(nsgcqt_plan plan, const float* x, float* coeffs, void* stream);

/* S: coeffs [batch][C] c64 -> x_out [batch][N] f32 (eq. 10). */
int nsgcqt_synthesise(nsgcqt_plan plan, const float* coeffs, float* x_out,
                      void* ws, size_t ws_bytes, void* stream);

/* Real adjoints (eqs. 13-14).
 *   NSGCQT_OP_ADJ_ANALYSIS : in = coefficient cotangent [batch][C] c64,
 *                            out = signal gradient [batch][N] f32
 *   NSGCQT_OP_ADJ_SYNTHESIS: in = signal cotangent [batch][N] f32,
 *                            out = coefficient gradient [batch][C] c64
 * EINVAL for any other op. */
int nsgcqt_adjoint(nsgcqt_plan plan, int op, const float* in, float* out,
                   void* ws, size_t ws_bytes, void* stream);

/* Number of slices J = ceil(n/H) + 1 a sliced plan produces for n samples. */
int64_t nsgcqt_sliced_count(nsgcqt_plan plan, int64_t n);

/* Sliced analysis of one signal x [n] f32 into coeffs [J][C] c64. */
int nsgcqt_sliced_analyse(nsgcqt_plan plan, const float* x, int64_t n, float* coeffs,
                          void* ws, size_t ws_bytes, void* stream);

/* Sliced synthesis: overlap-add of the slices' syntheses, cropped to n
 * samples, coeffs [J][C] c64 -> x_out [n] f32. */
int nsgcqt_sliced_synthesise(nsgcqt_plan plan, const float* coeffs, int64_t n, float* x_out,
                             void* ws, size_t ws_bytes, void* stream);

/* Profiling hook. While `events` is non-NULL, every compute call on this
 * plan brackets its i-th kernel launch with events[2i] (before) and
 * events[2i+1] (after), both recorded on the stream the kernel runs on
 * (the call's stream, or a plan side stream when the call's band phase
 * fans out), for as many pairs as given (hipEvent_t handles created by the
 * caller; NULL entries are skipped, so single kernels can be timed alone).
 * The kernel order is that of nsgcqt_stage_info. A NULL `events` stops recording. The setting
 * is plan state: do not combine it with concurrent calls on the same plan. */
int nsgcqt_set_stage_events(nsgcqt_plan plan, void* const* events, int n_events);

/* Kernels one call of `op` enqueues, in enqueue order: returns their count
 * (>= 0) or a negative status. For i in range, writes the kernel's name and
 * the algorithmic bytes one launch must move (inputs read once, outputs
 * written once; persistent tables excluded). name/alg_bytes may be NULL.
 * For a sliced plan (Sec. 4 slicing) the list is that of one chunk of
 * slices_per_chunk slices, which a sliced call repeats per chunk (the last
 * chunk may hold fewer slices): NSGCQT_OP_ANALYSE gives the analysis chain,
 * NSGCQT_OP_SYNTHESISE the synthesis chain followed by the overlap-add of the
 * chunk's slices; other ops are EINVAL. Stage events then bracket the
 * kernels of the first chunk. */
int nsgcqt_stage_info(nsgcqt_plan plan, int op, int i, char* name, size_t name_cap,
                      double* alg_bytes);

/* Message of the last failing call on this thread ("" if none). */
const char* nsgcqt_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* NSGCQT_H */
