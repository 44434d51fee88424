/*
 * lapsum.h - exact-budget LapSum soft top-k ("Fast LapSum") on AMD Instinct
 * MI355X (gfx950).  C ABI of liblapsum.so.
 *
 * The operator (paper: "Fast LapSum: Exact Differentiable Top-k at Million
 * Scale", Eq. (1) and Suppl. A): given scores r in R^n, a budget k in (0, n)
 * and a temperature alpha < 0 (t = -alpha), find the threshold b with
 *
 *     LapSum(b) = sum_i sigma((b - r_i) / alpha) = k,
 *
 * sigma being the Laplace CDF (sigma(u) = e^u / 2 for u <= 0, 1 - e^{-u} / 2
 * for u > 0, Eq. (3)), and return p_i = sigma((b - r_i) / alpha).  LapSum is
 * strictly decreasing in b, so b is unique.  Larger scores get larger p, and
 * sum_i p_i = k exactly up to rounding.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers are DEVICE pointers (memory of the current HIP device) unless a
 *    comment says otherwise.  The caller owns all memory; the library never
 *    allocates device memory and keeps no state across calls (beyond a
 *    small pinned host buffer per host thread, see the bracketed forward).
 *  - Arrays are row-major [batch, n] and contiguous; k and alpha are shared
 *    by all rows.  Indices are int32 and count within a row.
 *  - Each call validates its scalar arguments on the host, then enqueues
 *    kernels on `stream` and returns.  Results are valid once the stream has
 *    synchronised.  lapsum_forward_bracketed additionally waits on `stream`
 *    once per row to read the bracket certificate (see there).
 *  - Errors are returned as lapsum_status codes; no call aborts or throws.
 *    On an error nothing has been enqueued, except LAPSUM_ERR_HIP, which can
 *    follow earlier launches of the same call.
 *  - Scores must be finite; NaN or infinite scores give unspecified outputs
 *    (they are not scanned for).
 *  - workspace: caller-owned scratch of at least the size the matching
 *    *_workspace_size function returns, aligned to 256 bytes.  Its content
 *    on entry does not matter.  Two calls that overlap in time (different
 *    streams) must use different workspaces.
 *  - Only gfx950 devices are accepted (LAPSUM_ERR_DEVICE otherwise).
 */
#ifndef LAPSUM_H
#define LAPSUM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lapsum_status {
    LAPSUM_OK = 0,
    LAPSUM_ERR_INVALID_ARG = 1, /* null required pointer; batch < 1; n < 1 or
                                   n > 2^31 - 1; k not in (0, n); alpha not a
                                   finite negative number; bracketed: K < 2 or
                                   K > n, z not finite and > 0, m_capacity < 1,
                                   unknown flag bits */
    LAPSUM_ERR_WORKSPACE = 2,   /* workspace NULL, too small, or not 256-byte
                                   aligned */
    LAPSUM_ERR_HIP = 3,         /* a HIP runtime call or kernel launch failed */
    LAPSUM_ERR_DEVICE = 4       /* the current device is not gfx950 */
} lapsum_status;

/* Static description of a status code (host memory, never freed). */
const char* lapsum_status_string(int status);

/* ------------------------------------------------------------------------
 * Full-sort forward (paper §1, §3, Suppl. A): sort each row descending, one
 * prefix/suffix exponential scan gives the node curve LapSum(r_(i)), an index
 * lookup finds the interval holding b and the two-exponential equation on it
 * is solved in closed form; then the Laplace CDF is evaluated for every score
 * in the original order.
 *
 *   scores   [batch, n] float32, input.
 *   k        budget, 0 < k < n (real; the same for every row).
 *   alpha    temperature, alpha < 0.
 *   p        [batch, n] float32, output p_i = sigma((b - r_i) / alpha).
 *   b        [batch] float64, output threshold per row.
 *   perm_out NULL, or [batch, n] int32 output: perm_out[row][i] = original
 *            index of the i-th largest score of the row.  Ties in value are
 *            ordered by the order-preserving uint32 key of the float (so
 *            +0.0 precedes -0.0) and then by ascending original index.
 *            Asking for it makes the sort carry indices (slower).
 * Rows with n <= 32768 are solved by one workgroup per row entirely on chip,
 * except a batch of one row longer than 16384, which is faster through the
 * device-wide sort and scan; longer rows use the device-wide path, one row
 * after another.  The workspace size depends on batch for that reason.
 * ------------------------------------------------------------------------ */
size_t lapsum_forward_workspace_size(int64_t batch, int64_t n, int with_perm);

int lapsum_forward(const float* scores, int64_t batch, int64_t n, double k,
                   double alpha, float* p, double* b, int32_t* perm_out,
                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * lapsum_forward_noalloc: lapsum_forward for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and outputs, with the workspace taken from a
 * device array of LAPSUM_NOALLOC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends.  The call makes no
 * allocation (its first call on a device only looks the array's address
 * up).  The caller still passes scores and outputs.
 *
 *   arguments as lapsum_forward, without workspace
 *   LAPSUM_ERR_WORKSPACE when lapsum_forward_workspace_size(batch, n,
 *   perm_out != NULL) exceeds LAPSUM_NOALLOC_SCRATCH_BYTES (rows of up to
 *   32768 scores need none; one long row fits up to 3,943,808 scores with
 *   perm_out and 7,443,072 without).
 * All calls on one GPU share its array: calls that overlap in time on one
 * GPU (different streams, or host threads) race and must not be issued.
 * ------------------------------------------------------------------------ */
#define LAPSUM_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)

int lapsum_forward_noalloc(const float* scores, int64_t batch, int64_t n,
                           double k, double alpha, float* p, double* b,
                           int32_t* perm_out, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Backward: the analytical vector-Jacobian product of Eq. (5),
 *
 *   grad_r = f * (g - <g, q>),  q = f / sum_j f_j,
 *   f_i = exp(-|b - r_i| / t) / (2 t) = min(p_i, 1 - p_i) / t,
 *
 * evaluated from the forward's p (the two forms of f are equal for the
 * Laplace CDF).  One reduction of (sum f, sum f g) per row, then one
 * element-wise pass.  When sum f is zero in floating point (every p is
 * exactly 0 or 1) grad_r is zero.
 *
 *   grad_p  [batch, n] float32, upstream gradient dL/dp.
 *   p       [batch, n] float32, the forward output for the same k, alpha.
 *   b       [batch] float64 or NULL; not read by this p-form (accepted so
 *           that callers can pass the forward's outputs unchanged).
 *   alpha   the forward's temperature.
 *   grad_r  [batch, n] float32, output dL/dr.
 *   grad_k, grad_alpha
 *           [batch] float64 device memory each, or NULL: the gradients of
 *           L with respect to the budget k and the temperature alpha, which
 *           the adversarial attack of §5 trains along with the input (the
 *           paper gives no formula; these follow from differentiating
 *           Eq. (1) implicitly).  With s_i = min(p_i, 1 - p_i) and
 *           u_i = (r_i - b)/t (recovered from p_i: |u_i| = -ln(2 s_i),
 *           negative where p_i <= 1/2),
 *             dL/dk     = sum s g / sum s  (= <g, q>),
 *             dL/dalpha = (sum s g u - (sum s u / sum s) sum s g) / t,
 *           both 0 when sum s is zero.  Requesting either adds the two
 *           extra sums to the same reduction; NULL for both leaves the pass
 *           as it is.
 * ------------------------------------------------------------------------ */
size_t lapsum_backward_workspace_size(int64_t batch, int64_t n);

int lapsum_backward(const float* grad_p, const float* p, const double* b,
                    int64_t batch, int64_t n, double alpha, float* grad_r,
                    double* grad_k, double* grad_alpha,
                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Hard top-k mask for the straight-through estimator of Suppl. "Straight-
 * Through Estimator": m_i = 1 when r_i is among the k largest scores of its
 * row, else 0, so that sum_i m_i = k.  It is formed from the descending
 * order that lapsum_forward returns in perm_out (equal scores ordered by
 * index, so exactly k ones even with ties).  The estimator itself,
 * m^ = p + sg(m - p), is assembled by the caller's autodiff.
 *
 *   perm   [batch, n] int32, a descending order per row (lapsum_forward's
 *          perm_out).  Entries outside [0, n) are skipped; positions that no
 *          entry names are left unchanged.
 *   k      integer count of ones per row, 0 <= k <= n.
 *   mask   [batch, n] float32 output.
 * ------------------------------------------------------------------------ */
int lapsum_topk_mask(const int32_t* perm, int64_t batch, int64_t n, int64_t k,
                     float* mask, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Comparators (not part of the operator): the two methods the paper measures
 * Fast LapSum against, so that its speed and budget claims can be checked on
 * this device.
 *
 * lapsum_bisect_forward: the per-query bisection baseline of §5 ("Speed"),
 * the pattern of the original LapSum implementation: one thread per row runs
 * `steps` bisection steps on LapSum(b) = k, each re-summing all n Laplace-CDF
 * terms, in float32 throughout (scores, midpoints, terms and the running
 * sum), from lo = min r - t (ln(n / (2(n - k)))^+ + 1) and
 * hi = max r + t (ln(n / (2k))^+ + 1); b = the last midpoint, and p as in
 * lapsum_forward.  The paper runs 60 steps.
 *   scores, k, alpha, p, b   as in lapsum_forward (b: the float32 midpoint
 *                            widened to float64)
 *   steps                    0..200
 *
 * lapsum_dftopk_forward / _backward: DFTopK (§2; Suppl. "Comparison with
 * DFTopK"): the threshold fixed at c = (r_(k) + r_(k+1)) / 2, the midpoint of
 * the k-th and (k+1)-th largest scores of the row (equal scores ranked by
 * index as in lapsum_forward's perm_out), and the logistic step
 * p_i = 1 / (1 + e^{-(r_i - c)/t}) (the paper names a smooth step; its
 * Table budget value for DFTopK, a mass 3.46 k at alpha = -1, is the
 * logistic one).  The budget is not exact: sum p drifts from k.  The
 * backward is the VJP of that map: grad_i = g_i s_i / t with
 * s_i = p_i (1 - p_i), minus (1/(2t)) sum_j g_j s_j at the two boundary
 * scores (c moves by 1/2 with each).  Rows are processed one after another
 * (one device-wide sort each).
 *   k       integer, 1 <= k < n (n >= 2)
 *   c       [batch] float64 output: the thresholds
 *   pair    [batch, 2] int32: forward output, backward input: the indices
 *           of r_(k) and r_(k+1) in each row
 *   workspace  lapsum_dftopk_workspace_size(batch, n) bytes, 256-aligned
 * ------------------------------------------------------------------------ */
int lapsum_bisect_forward(const float* scores, int64_t batch, int64_t n,
                          double k, double alpha, int32_t steps, float* p,
                          double* b, hipStream_t stream);

size_t lapsum_dftopk_workspace_size(int64_t batch, int64_t n);

int lapsum_dftopk_forward(const float* scores, int64_t batch, int64_t n,
                          int64_t k, double alpha, float* p, double* c,
                          int32_t* pair, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);

int lapsum_dftopk_backward(const float* grad_p, const float* p,
                           const int32_t* pair, int64_t batch, int64_t n,
                           double alpha, float* grad_r, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Bracketed forward for very long rows (paper §4, Suppl. B, Suppl. C,
 * Algorithm 1, validated path of Suppl. D):
 *
 *  1. systematic sample of K kernel-noised scores,
 *     y_s = fl32(r[s * floor(n / K)] + noise[s]), s = 0..K-1 (the deployed
 *     sampler of §4), or with sample_idx the i.i.d. sample that the coverage
 *     theorem of Suppl. C assumes, y_s = fl32(r[sample_idx[s]] + noise[s]);
 *  2. ranks of Eq. (8) in IEEE float64: q = (n - k) / n,
 *     j = floor(K q - z sqrt(K q (1 - q))), l = ceil(K q + z sqrt(K q (1 - q)));
 *     a_L = y_(j), a_R = y_(l) (1-based order statistics; j < 1 gives
 *     a_L = -inf, l > K gives a_R = +inf);
 *  3. one pass over r: L = {r < a_L}, M = {a_L <= r < a_R}, R = {r >= a_R},
 *     the tail sums of Eq. (7) S_L = sum_L e^{-(a_L - r)/t},
 *     S_R = sum_R e^{-(r - a_R)/t}, the counts, and M gathered in index order;
 *  4. the scan of Suppl. A over M in descending order with the tails as
 *     carries gives LapSum(a_L) and LapSum(a_R); the bracket is certified when
 *     LapSum(a_R) <= k <= LapSum(a_L).  M is scanned in 2048 buckets of
 *     consecutive keys and only the bucket holding the root is sorted (all of
 *     M is sorted when m_idx_out is requested, or when that bucket holds more
 *     than 4096 scores); both give the same b;
 *  5. certified: b by the closed-form root (Suppl. B).  Not
 *     certified: the failing side is widened by one-sided doubling
 *     (LapSum(a_R) > k: a_L <- a_R, a_R <- a_R + 2 (a_R - a_L); LapSum(a_L) < k:
 *     a_R <- a_L, a_L <- a_L - 2 (a_R - a_L); float64 arithmetic on the
 *     float32 endpoints, rounded to float32) and steps 3-5 repeat.  After 3
 *     brackets, or when |M| > m_capacity, the row is solved by the full-sort
 *     path instead;
 *  6. p_i = sigma((b - r_i) / alpha) in the original order.  The pass of
 *     step 3 also keeps the band lo <= r < hi, lo = a_L - 105 t and
 *     hi = a_R + 18 t (rounded outwards to float32): for any b in a certified
 *     bracket, p is exactly 0 below the band and exactly 1 above it in
 *     float32, so step 6 writes p from the band and one bit per score
 *     without reading r again.  When t is so large against the spread of
 *     the scores that a quarter or more of the row's blocks cannot list
 *     their band, step 6 (and the backward from the saved band) streams the
 *     whole row instead; the values are the same.
 *
 * The result is the same b as lapsum_forward (the bracket only locates it).
 * The host waits on `stream` for each bracket attempt's record (set sizes
 * and certificate), so this call returns after every row's threshold is
 * known (the emit of step 6 may still be running).  In a batch without
 * m_idx_out the first brackets of up to 4 rows are enqueued before the
 * host waits for the first row's record, each with its own slice of the
 * workspace (lapsum_forward_bracketed_workspace_size counts the slices).
 * The first call on a host thread allocates a small pinned host buffer
 * that the library keeps.
 *
 *   K           sample size, 2 <= K <= n.
 *   z           bracket half-width in standard deviations (the paper uses
 *               5.16), finite and > 0.
 *   noise       NULL, or [K] float32 Laplace(0, |alpha|) draws shared by all
 *               rows (the cached kernel noise of §4 and Algorithm 1).  NULL:
 *               the library draws the table itself from `seed`, the same
 *               draws lapsum_bracket_noise(seed, K, alpha) writes (they are
 *               formed inside the sample pass, so no table is stored).
 *   seed        the default noise's seed; ignored when noise is given.
 *   sample_idx  NULL (systematic sample), or [K] int32 indices drawn
 *               uniformly from [0, n) by the caller, shared by all rows
 *               (i.i.d. sample); entries outside [0, n) are clamped to it.
 *   m_capacity  largest |M| the workspace holds, >= 1.
 *   flags       0, or LAPSUM_FLAG_FULL_SORT to skip the bracket and solve
 *               by the full-sort path (same outputs; info->fell_back = 1).
 *   p, b        as in lapsum_forward.
 *   info        NULL, or [batch] lapsum_bracket_info in HOST memory, filled
 *               with the last attempt's record.
 *   m_idx_out   NULL, or [batch, m_capacity] int32: the original indices of
 *               the final M in descending order (ties by ascending index),
 *               -1 after the first n_M entries.  Rows that fell back to the
 *               full sort get all -1.  Asking for it makes the M sort carry
 *               indices.
 *   band        NULL, or device memory of at least lapsum_band_size(batch, n)
 *               bytes, 256-byte aligned (band_bytes its size): receives the
 *               band of each row with its p, for lapsum_backward_band.  Its
 *               content is private to the library; it is valid once the
 *               call's work on `stream` has completed and until the caller
 *               reuses the memory.
 * ------------------------------------------------------------------------ */
#define LAPSUM_FLAG_FULL_SORT 1u

typedef struct lapsum_bracket_info {
    float a_L, a_R;        /* final bracket, +-INFINITY when unbounded */
    int64_t j, l;          /* 1-based ranks of the first bracket (Eq. (8)) */
    int64_t n_L, n_M, n_R; /* set sizes of the last attempt */
    double T_L, T_R;       /* tail sums S_L, S_R of the last attempt */
    double lap_aL, lap_aR; /* certificate values LapSum(a_L), LapSum(a_R) */
    int32_t attempts;      /* brackets tried, 1..3 (0 with the flag) */
    int32_t fell_back;     /* 1 if the row was solved by the full sort */
    int32_t m_overflow;    /* 1 if |M| exceeded m_capacity */
    int32_t reserved;
} lapsum_bracket_info;

size_t lapsum_forward_bracketed_workspace_size(int64_t batch, int64_t n,
                                               int64_t K, int64_t m_capacity,
                                               int with_m_idx);

size_t lapsum_band_size(int64_t batch, int64_t n);

int lapsum_forward_bracketed(const float* scores, int64_t batch, int64_t n,
                             double k, double alpha, int64_t K, double z,
                             const float* noise, uint64_t seed,
                             const int32_t* sample_idx,
                             int64_t m_capacity, uint32_t flags, float* p, double* b,
                             lapsum_bracket_info* info, int32_t* m_idx_out,
                             void* band, size_t band_bytes,
                             void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* ------------------------------------------------------------------------
 * The bracket's default kernel noise (§4: the sample is a strided view plus
 * cached Laplace kernel noise; Algorithm 1 draws it once): draw s of seed
 * `seed`, s = 0..K-1, is
 *
 *   z = the (s+1)-th output of SplitMix64 started at state `seed` (Steele,
 *       Lea and Flood, "Fast splittable pseudorandom number generators",
 *       OOPSLA 2014): x = seed + (s+1) 0x9E3779B97F4A7C15 (mod 2^64),
 *       z = (x ^ (x >> 30)) 0xBF58476D1CE4E5B9, z = (z ^ (z >> 27))
 *       0x94D049BB133111EB, z = z ^ (z >> 31);
 *   u = (2 (z >> 12) + 1) 2^-53, strictly inside (0, 1);
 *   eps_s = t ln(2u) for u < 1/2, -t ln(2(1 - u)) otherwise (the Laplace
 *       inverse CDF, t = -alpha), in float64, rounded to float32.
 *
 * A counter-based generator: the same (seed, s) gives the same draw on
 * every call, so the table needs no storage.  This call writes the table
 * that lapsum_forward_bracketed uses when it is given noise == NULL.
 *   out   [K] float32 device memory, 1 <= K <= 2^31 - 1.
 * ------------------------------------------------------------------------ */
int lapsum_bracket_noise(uint64_t seed, int64_t K, double alpha, float* out,
                         hipStream_t stream);

/* ------------------------------------------------------------------------
 * Backward from a saved band: the same vector-Jacobian product as
 * lapsum_backward (Eq. (5)), for the p of a lapsum_forward_bracketed call
 * that was given `band`.  f = min(p, 1 - p) / t is zero outside the band, so
 * the sums of f and f g visit the band only (g is read where f != 0) and
 * grad_r is written densely, zero outside the band, without reading p.
 * Blocks of the row whose band did not fit the library's lists, and rows
 * that fell back to the full sort, are computed from p and grad_p directly.
 *
 *   grad_p, p, alpha, grad_r   as in lapsum_backward (p: the forward's output)
 *   grad_k, grad_alpha         as in lapsum_backward; u_i is taken from the
 *                              saved score for band members and from p_i in
 *                              blocks computed from p
 *   band, band_bytes           the forward's band, unchanged since; a band
 *                              saved for another row length is detected and
 *                              the dense form used instead
 * INVALID_ARG also when band is NULL, smaller than lapsum_band_size(batch, n)
 * or not 256-byte aligned.
 * ------------------------------------------------------------------------ */
size_t lapsum_backward_band_workspace_size(int64_t batch, int64_t n);

int lapsum_backward_band(const float* grad_p, const float* p, const void* band,
                         size_t band_bytes, int64_t batch, int64_t n,
                         double alpha, float* grad_r, double* grad_k,
                         double* grad_alpha, void* workspace,
                         size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Diagnostics: per-kernel timing with HIP events.  Off by default.  While
 * on, every kernel the library launches is bracketed by two events recorded
 * on the launch stream (this adds a little host work per launch).  Not
 * thread-safe: start, run, stop from one host thread.
 *
 *   lapsum_profile_start()   clears previous records and turns recording on
 *   lapsum_profile_stop()    turns it off, waits for the recorded events and
 *                            aggregates them by kernel name; returns the
 *                            number of distinct kernels (or -LAPSUM_ERR_HIP)
 *   lapsum_profile_entry(i, name, name_len, launches, total_ms)
 *                            the i-th aggregate: name (NUL-terminated, host
 *                            buffer of name_len bytes), launch count and
 *                            summed duration in milliseconds
 * ------------------------------------------------------------------------ */
int lapsum_profile_start(void);
int lapsum_profile_stop(void);
int lapsum_profile_entry(int i, char* name, size_t name_len, int64_t* launches,
                         double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* LAPSUM_H */
