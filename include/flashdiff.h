/*
 * flashdiff.h -- C ABI of the diffusion-map kernel library for MI355X (gfx950).
 *
 * The library applies the Gaussian affinity K_ij = exp(-beta ||x_i - x_j||^2)
 * of a point cloud X (N x D) to blocks of vectors without ever forming the
 * N x N matrix, builds the Coifman-Lafon normalisation from it, and runs a
 * block Lanczos eigensolver and a warm-started (n, beta) continuation on top.
 * Paper: FlashDiffusion, Sec. 2 ("FlashDiffusion Algorithm").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Device pointers are caller-owned HIP device memory on the current device.
 *    Host pointers are marked "host".  The library allocates no device memory:
 *    every temporary lives in the caller's workspace `ws` of `ws_bytes` bytes,
 *    at least fd_workspace_size(...) bytes, 256-byte aligned.
 *  - Matrices are row-major.  X is N x D with leading dimension ldx >= D
 *    (elements, not bytes); V, Y, eigenvector blocks are N x b with their own
 *    leading dimensions.  X holds float32 (FD_F32) or bfloat16 bit patterns
 *    (FD_BF16); all other floating-point arrays are float32 unless stated.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream).
 *    fd_kernel_matmul and fd_degree are asynchronous.  fd_block_lanczos and
 *    fd_continuation synchronise `stream` at every restart cycle to read a few
 *    scalars back, and return after all their work has completed.
 *  - Every function returns an fd_status and never throws.  On a non-OK status
 *    fd_last_error() returns a thread-local message; output contents are then
 *    unspecified unless the status says otherwise.
 *  - Centring: the method is stated for centred observations (Sec. 2.1, eq.
 *    rbf_gram), and the Gram-form evaluation loses accuracy far from the
 *    origin.  For float32 X the library centres on the device (column means
 *    in float64, subtracted before the exponent contraction; the kernel is
 *    translation invariant, so results are unchanged up to rounding);
 *    bfloat16 X is used as given and should be centred by the caller.
 *  - Accuracy envelope (float32 X): K V to 1e-5 relative (measured 1e-7 to
 *    4e-6) while B = beta log2(e) max_i ||x_i - mean||^2 <= 200; above 64 the
 *    feature widths whose fast exponent layout drops the third offset piece
 *    (13 < D <= 30, 32 < D <= 62) switch to one that keeps it.  Beyond
 *    B = 200 the dropped fourth-order piece products can reach the 1e-5 bar
 *    (1.1e-5 measured at B = 400, D = 30).
 *  - Exponent range (float32 X): the offsets and the scaled coordinates enter
 *    the contraction as float16 pieces, so B above 65488 cannot be formed at
 *    all, nor (when beta is so small that the coordinate scale stops at
 *    2^-12) coordinates whose scaled pieces pass 65504.  There the
 *    asynchronous entry points fill their outputs with NaN (fd_degree_dyadic:
 *    when its largest bandwidth is beyond), fd_block_lanczos and
 *    fd_continuation return FD_ERR_UNSUPPORTED (the continuation's earlier
 *    steps stay valid), and the flow ends its sweep before such a probe.
 *  - Non-finite X: every entry point scans X on the device first.  The
 *    asynchronous ones (fd_kernel_matmul, fd_kernel_matmul_noalloc, fd_degree,
 *    fd_degree_dyadic) then fill all their outputs with NaN; the eigensolver,
 *    continuation and flow entry points return FD_ERR_INVALID_ARG before any
 *    other work.
 */
#ifndef FLASHDIFF_H
#define FLASHDIFF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fd_status {
  FD_OK = 0,
  FD_ERR_INVALID_ARG = 1,    /* bad size, pointer, or parameter value */
  FD_ERR_UNSUPPORTED = 2,    /* valid request the library does not implement */
  FD_ERR_WORKSPACE = 3,      /* workspace missing, too small or misaligned */
  FD_ERR_HIP = 4,            /* a HIP runtime or launch error (message has it) */
  FD_ERR_NOT_CONVERGED = 5,  /* eigensolver stopped early; outputs hold best Ritz pairs */
  FD_ERR_PERRON_WALL = 6     /* continuation stopped at the precision wall */
} fd_status;

typedef enum fd_dtype {
  FD_F32 = 0,   /* X in float32 */
  FD_BF16 = 1   /* X as bfloat16 bit patterns (uint16) */
} fd_dtype;

typedef enum fd_op {
  FD_OP_KERNEL_MATMUL = 0,
  FD_OP_DEGREE = 1,
  FD_OP_BLOCK_LANCZOS = 2,
  FD_OP_CONTINUATION = 3,
  FD_OP_BETA_FLOW = 4,
  FD_OP_DEGREE_DYADIC = 5
} fd_op;

/* Options of the block Lanczos eigensolver (Sec. 2.3, first paragraph: block
 * implicitly restarted Lanczos; realised as thick-restart block Lanczos with
 * full reorthogonalisation).  fd_lanczos_default_opts fills the defaults. */
typedef struct fd_lanczos_opts {
  double tol;               /* converged when ||M phi - theta phi||_2 <= tol (||M||_2 = 1). Default 1e-5 */
  int32_t max_restarts;     /* restart cycles before FD_ERR_NOT_CONVERGED. Default 200 */
  int32_t max_basis_blocks; /* basis capacity in blocks of b (0 = automatic: four times the first
                               cycle's width, at most 1024 columns).  The first restart cycle
                               grows the basis to k + keep rounded up to whole blocks plus as
                               many again (at least 2 blocks), then runs Rayleigh-Ritz and a
                               thick restart; a cycle that converged few new leading pairs
                               doubles the next cycle's width, up to the capacity.  After a warm
                               start the first cycle is a single block */
  int32_t keep;             /* Ritz vectors kept at restart beyond k (-1 = automatic: k, at least
                               b, as far as k + keep + b fits the capacity) */
  int32_t max_matvecs;      /* stop after this many block products (0 = no limit). A run that
                               stops this way returns FD_ERR_NOT_CONVERGED with valid Ritz pairs */
  int32_t verbose;          /* non-zero: one progress line per restart cycle on stderr */
  uint64_t seed;            /* seed of the counter-based generator for start/fill vectors */
} fd_lanczos_opts;

/* Per-solve report (host memory). */
typedef struct fd_lanczos_info {
  int32_t restarts;         /* restart cycles run */
  int32_t block_matvecs;    /* applications of M to a block of b vectors */
  int32_t nconv;            /* leading Ritz pairs with residual <= tol */
  int32_t wall;             /* 1 when g_P <= kappa_P * eta, kappa_P = 10 and eta of X's dtype
                               (fp32 1e-7, bf16 8e-3) (Sec. 2.3, eq. perronwall and its footnote) */
  double gap_perron;        /* g_P = (theta_0 - theta_1) / |theta_0| */
  double s_off;             /* S_off = sum_{i != j} K_ij = sum(q) - N (Sec. 2.3) */
  double max_residual;      /* largest residual among the k returned pairs */
  double seconds;           /* wall time of the call, host clock */
} fd_lanczos_info;

/* Fill *opts with the defaults listed above. */
void fd_lanczos_default_opts(fd_lanczos_opts* opts);

/* Bytes of workspace an entry point needs.
 *   op = FD_OP_KERNEL_MATMUL: Nr output rows, Nc columns, D, b; k ignored.
 *   op = FD_OP_DEGREE:        Nr = Nc = N, D; b, k ignored.
 *   op = FD_OP_DEGREE_DYADIC: Nr = Nc = N, D; b, k ignored.
 *   op = FD_OP_BLOCK_LANCZOS: Nr = Nc = N, D, b, k, opts (NULL = defaults).
 *   op = FD_OP_BETA_FLOW:     Nr = Nc = N, D, b, k, opts (NULL = defaults); also the
 *                             size for fd_beta_flow_cascade.
 *   op = FD_OP_CONTINUATION:  Nr = largest n of the schedule, Nc = number of steps,
 *                             D, b, k (<= 64), opts.
 * Returns 0 for arguments the entry point would reject. */
size_t fd_workspace_size(fd_op op, int64_t Nr, int64_t Nc, int64_t D, int64_t b, int64_t k,
                         const fd_lanczos_opts* opts);

/* Fused Gaussian-kernel block product (Sec. 2.1 eq. matmat; Sec. 2.2 eq. tiled_rbf):
 *
 *     Y = diag(sl) K(Xr, Xc) diag(sr) V,   K_ij = exp(-beta ||xr_i - xc_j||^2),
 *
 * evaluated tile by tile in the Gram form of eq. rbf_gram (row norms plus a
 * matrix-core contraction), exponentiated and multiplied into V on chip.
 *   Xr  : Nr x D rows (device, dtype xt, ldx);  Xc : Nc x D columns (same D, ldx, xt).
 *         When Xr == Xc (the same array; the shorter set is then a prefix of the
 *         longer) every K_ii with i < min(Nr, Nc) is taken as exactly 1.
 *   beta: >= 0 (beta = 0 gives K = ones).
 *   sl  : Nr scale of output rows, or NULL for ones.  sr : Nc scale of V rows, or NULL.
 *   V   : Nc x b (device, ldv >= b), 1 <= b <= 64.   Y : Nr x b output (device, ldy >= b).
 *         Y must not overlap V, sl, sr or X.
 * Float32 accumulation.  Deterministic: repeated calls give identical bits. */
fd_status fd_kernel_matmul(const void* Xr, int64_t Nr, const void* Xc, int64_t Nc, int64_t D,
                           int64_t ldx, fd_dtype xt, float beta, const float* sl, const float* sr,
                           const float* V, int64_t b, int64_t ldv, float* Y, int64_t ldy,
                           void* ws, size_t ws_bytes, void* stream);

/* Allocation-free variant of fd_kernel_matmul, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments and result as
 * fd_kernel_matmul (the same kernels, bit for bit), without the workspace: the
 * temporaries live in a scratch array built into the library,
 * fd_kernel_matmul_noalloc_limit() bytes (256 MiB) per device, which each
 * device holds from the library's load until the process ends.  A problem
 * whose temporaries do not fit returns FD_ERR_WORKSPACE (for example, b = 16
 * fits up to about 2^18 points with D <= 12).  The call allocates nothing.
 * Every call on one device shares that device's scratch, and a call only
 * relies on what it writes there itself: calls that overlap in time on one
 * device (several streams or threads) race and give wrong results, so
 * serialise them.  Asynchronous on `stream`, like fd_kernel_matmul. */
fd_status fd_kernel_matmul_noalloc(const void* Xr, int64_t Nr, const void* Xc, int64_t Nc,
                                   int64_t D, int64_t ldx, fd_dtype xt, float beta,
                                   const float* sl, const float* sr, const float* V, int64_t b,
                                   int64_t ldv, float* Y, int64_t ldy, void* stream);

/* Bytes of the built-in scratch of fd_kernel_matmul_noalloc. */
size_t fd_kernel_matmul_noalloc_limit(void);

/* Normalisation passes (Sec. 2.1, the two "entry fee" applications):
 *     q = K 1;  w = q^-alpha;  d = w * (K w);  s = w * d^-1/2,
 * so that M = diag(s) K diag(s) and P = diag(d)^-1 diag(w) K diag(w).
 * With alpha = 0 the second application is skipped (d = q).
 *   X: N x D (device).  beta > 0.  0 <= alpha <= 1.
 *   q, d, s: N-vectors (device) or NULL each.
 *   s_off: one double (device) receiving sum(q) - N = sum_{i != j} K_ij (Sec. 2.3), or NULL. */
fd_status fd_degree(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx, float beta,
                    float alpha, float* q, float* d, float* s, double* s_off, void* ws,
                    size_t ws_bytes, void* stream);

/* Normalisation vectors of a dyadic bandwidth ladder beta_l = beta0 2^l,
 * l = 0 .. nbeta - 1 (Sec. 2.3, dyadic continuation): level l holds what
 * fd_degree returns at beta_l, up to rounding.  The kernel at 2 beta is the
 * entrywise square of the kernel at beta (eq. kernel), so on float32 inputs
 * with alpha > 0 the second pass of level l also sums K(beta_l)^2 along rows
 * and columns, which is level l + 1's q = K(beta_{l+1}) 1: every level after
 * the first takes one pass over the kernel instead of two.  Other inputs run
 * fd_degree's passes level by level.
 *   X: N x D (device).  beta0 > 0 with beta0 2^(nbeta-1) finite; 1 <= nbeta <= 32;
 *   0 <= alpha <= 1.
 *   q, d, s: nbeta x N floats each (device; level l at offset l N), or NULL each.
 *   s_off: nbeta doubles (device), sum(q_l) - N per level, or NULL.
 *   Workspace: fd_workspace_size(FD_OP_DEGREE_DYADIC, N, N, D, 0, 0, NULL).
 * Asynchronous on `stream`. */
fd_status fd_degree_dyadic(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                           float beta0, int32_t nbeta, float alpha, float* q, float* d, float* s,
                           double* s_off, void* ws, size_t ws_bytes, void* stream);

/* Top-k eigenpairs of M = diag(s) K diag(s) by thick-restart block Lanczos
 * (Sec. 2.3, first paragraph; Sec. 2.1 eq. symmetric), including the Perron
 * pair theta_0 = 1.  Computes the normalisation itself (fd_degree) and then
 * applies M to blocks of b vectors, one fused product per block.
 * A solve stops early at the Perron wall (eq. perronwall): when the Perron pair
 * has converged and the Ritz gap (theta_0 - theta_1) / theta_0, an upper bound
 * of the true gap, is at or below kappa_P eta (eta of X's dtype), the leading
 * eigenspace is not resolvable in that precision; info->wall is then 1 and
 * the status FD_ERR_NOT_CONVERGED unless all k pairs had converged.
 *   X: N x D (device).  beta > 0, 0 <= alpha <= 1, 1 <= b <= 64, 1 <= k <= N.
 *   V0: optional warm start, N x k0 (device, ldv0 >= k0); NULL or k0 = 0 for a
 *       seeded random start.  Interpreted as Markov right eigenvectors psi
 *       (warm_is_psi = 1: converted with the new d^1/2) or as eigenvectors of M.
 *   evals: k doubles (host), descending.  evecs: N x k (device, ld k) orthonormal
 *       eigenvectors phi of M.  psi: N x k (device, ld k) Markov right eigenvectors
 *       d^-1/2 phi (last paragraph of Sec. 2.3), or NULL.
 *   residuals: k doubles (host) or NULL.  info: host report or NULL.
 * Returns FD_ERR_NOT_CONVERGED (outputs valid, info->nconv < k) when the restart
 * or product budget runs out. */
fd_status fd_block_lanczos(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                           float beta, float alpha, int64_t b, int64_t k, const float* V0,
                           int64_t k0, int64_t ldv0, int32_t warm_is_psi,
                           const fd_lanczos_opts* opts, double* evals, float* evecs, float* psi,
                           double* residuals, fd_lanczos_info* info, void* ws, size_t ws_bytes,
                           void* stream);

/* Warm-started (n, beta) ladder (Sec. 1, last paragraph; Sec. 2.3, dyadic
 * continuation with warm starts and the Perron wall of eq. perronwall).
 * Step t solves for the top-k eigenpairs on the prefix X[0:n_t] at beta_t.
 * Its start is the previous step's Markov eigenvectors psi: unchanged when
 * n_t equals the previous n, extended by the Nystrom formula (one rectangular
 * fused product over the previous prefix) when n_t grows; when n_t grows the
 * start is taken from the last step solved at n_{t-1} whose beta equals beta_t
 * if one exists, else the previous step.
 *   n_steps: nsteps prefix sizes (host), non-decreasing, 2 <= n_t <= N.
 *   beta_steps: nsteps bandwidths (host), > 0.
 *   V0/k0: optional warm start for step 0 (Markov form, N x k0 device) or NULL.
 *   k: 1 <= k <= 64 (the Nystrom pass applies the kernel to k + 1 columns).
 *   evals: nsteps x k doubles (host).  evecs: n_last x k (device, ld k) eigenvectors of
 *   M at the last step run (its first n rows are written).  psi: the matching Markov
 *   eigenvectors (same layout) or NULL.
 *   per_step: nsteps reports (host) or NULL.
 *   stop_at_wall: when non-zero, stop after the first step whose Perron gap is at or
 *   below kappa_P * eta (eta of X's dtype, as in info->wall) and return FD_ERR_PERRON_WALL; evals of the steps run
 *   so far are valid and *steps_done tells how many ran.
 *   steps_done: host int64 or NULL.
 * Returns FD_ERR_NOT_CONVERGED when a step short of the Perron wall stopped
 * before its k pairs converged; a step at the wall (per_step[t].wall = 1, its
 * solve stopped as fd_block_lanczos describes) is reported, not failed. */
fd_status fd_continuation(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                          float alpha, const int64_t* n_steps, const float* beta_steps,
                          int64_t nsteps, int64_t b, int64_t k, const float* V0, int64_t k0,
                          int64_t ldv0, const fd_lanczos_opts* opts, double* evals,
                          float* evecs, float* psi, fd_lanczos_info* per_step,
                          int32_t stop_at_wall, int64_t* steps_done, void* ws, size_t ws_bytes,
                          void* stream);

/* ---- bandwidth selection by the beta-function flow (Sec. 2.3) ----
 *
 * Dyadic probes beta_0, 2 beta_0, 4 beta_0, ... on all N points.  Each probe
 * runs the normalisation and the top-k eigensolve of M (k includes the Perron
 * pair), warm-started from the previous probe's Markov eigenvectors, and
 * records
 *   S_off = sum_{i != j} K_ij,  g_P = (lambda_0 - lambda_1) / |lambda_0|,
 *   V_bias = median_j -log(lambda_j / lambda_0) over the k - 1 nontrivial pairs (eq. vbias),
 *   V_mach = (kappa_P eta / g_P)^p (eq. vmach),
 * and, once the next dyadic probe has run,
 *   n_eff = S_off(beta)^2 / (N S_off(2 beta)) (eq. neff),  V_stat = (n_eff V_bias)^-1/2 (eq. vstat),
 *   V = V_bias + V_stat + V_mach (eq. vtotal),  d_hat = -2 dlog S_off / dlog beta (eq. dhat).
 * A probe with g_P <= kappa_P eta (eq. perronwall) ends the sweep; the last
 * admissible probe is then the achieved bandwidth.  When three consecutive
 * complete probes have V falling then rising, with V_bias falling and V_stat
 * or V_mach rising between the outer two, a quadratic in log beta through the
 * three gives a vertex, which one more probe resolves (if that probe is past
 * the wall, the middle probe is taken).  When max_probes run out first, the
 * complete probe with the smallest V is taken.  beta_0 defaults to
 * min(0.1, 1 / (2 mean_i ||x_i - mean||^2)) from the centred data (eq. beta0). */
typedef struct fd_flow_opts {
  double beta_start;   /* <= 0: beta_0 of eq. beta0 */
  double eta;          /* precision scale of the kernel data; <= 0: by dtype (fp32 1e-7, bf16 8e-3) */
  double kappa;        /* kappa_P, default 10 */
  double p;            /* barrier exponent, default 6 */
  int32_t max_probes;  /* dyadic probes at most, default 24 (1..64) */
  int32_t reserved;
} fd_flow_opts;

typedef struct fd_flow_probe {
  double beta, s_off, gap_perron, v_bias, v_mach;
  double n_eff, v_stat, v_total, d_hat;  /* NaN until the next dyadic probe ran */
  double seconds;
  int32_t role;        /* 0 dyadic probe, 1 vertex probe, 2 solve at the selected bandwidth */
  int32_t admissible;  /* g_P > kappa_P eta */
  int32_t status;      /* status of the probe's eigensolve (FD_OK or FD_ERR_NOT_CONVERGED) */
  int32_t block_matvecs, nconv;
  int32_t level;       /* cascade level of the probe (0 for fd_beta_flow) */
} fd_flow_probe;

/* Why a sweep ended: a bracket of V_total (then the vertex probe), the Perron
 * wall, the probe budget, or the next dyadic bandwidth lies beyond the float32
 * path's exponent range (beta log2(e) max ||x - mean||^2 > 65488; not probed;
 * the bandwidth is chosen as on the budget). */
typedef enum fd_flow_exit {
  FD_FLOW_BRACKET = 0,
  FD_FLOW_WALL = 1,
  FD_FLOW_BUDGET = 2,
  FD_FLOW_RANGE = 3
} fd_flow_exit;

void fd_flow_default_opts(fd_flow_opts* o);

/* Runs the flow and returns the eigenpairs at the achieved bandwidth.
 *   X: N x D (device, dtype xt, ldx).  0 <= alpha <= 1, 1 <= b <= 64, 2 <= k <= N.
 *   fopts, opts: NULL = defaults.
 *   probes: host array of at least max_probes + 2 records; *nprobes (host) receives
 *     how many were written: the dyadic probes in order (a probe past the wall
 *     included), then the vertex probe and the solve at the selected bandwidth,
 *     each if it ran.
 *   beta_x (host): achieved bandwidth.  exit_reason (host): an fd_flow_exit.
 *   evals (host, k), evecs (device, N x k, ld k), psi (device or NULL): the
 *     eigenpairs at beta_x as in fd_block_lanczos.
 * Returns FD_ERR_NOT_CONVERGED (outputs valid) when the solve at beta_x stopped
 * before k pairs converged, FD_ERR_PERRON_WALL (records valid, nothing else)
 * when already the first probe is past the wall, FD_ERR_UNSUPPORTED
 * (exit_reason FD_FLOW_RANGE, nothing else) when already the first bandwidth
 * is beyond the exponent range. */
fd_status fd_beta_flow(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx, float alpha,
                       int64_t b, int64_t k, const fd_flow_opts* fopts,
                       const fd_lanczos_opts* opts, fd_flow_probe* probes, int64_t* nprobes,
                       double* beta_x, int32_t* exit_reason, double* evals, float* evecs,
                       float* psi, void* ws, size_t ws_bytes, void* stream);

/* Precision cascade of the flow (Sec. 2.3, last paragraph): the same points
 * supplied in several data types, lowest precision first.  Level 0 runs the
 * flow of fd_beta_flow on Xs[0] (from beta_start, or beta_0 of eq. beta0);
 * each later level runs it on Xs[l] starting at the previous level's achieved
 * bandwidth, its first probe warm-started from the previous level's Markov
 * eigenvectors.  Each level uses the eta of its own data type (fp32 1e-7,
 * bf16 8e-3) unless fopts->eta > 0 fixes one for all.  The achieved bandwidth
 * and the eigenpairs are those of the last level.
 *   Xs, xts, ldxs: nlevels (1..4) device arrays of the same N x D points, their
 *     dtypes and leading dimensions (host arrays of pointers / values).
 *   probes: host array of at least nlevels * (max_probes + 2) records, each
 *     tagged with its level; other arguments and returns as fd_beta_flow
 *     (FD_ERR_PERRON_WALL when the first probe of any level is past the wall). */
fd_status fd_beta_flow_cascade(const void* const* Xs, const fd_dtype* xts, const int64_t* ldxs,
                               int32_t nlevels, int64_t N, int64_t D, float alpha, int64_t b,
                               int64_t k, const fd_flow_opts* fopts,
                               const fd_lanczos_opts* opts, fd_flow_probe* probes,
                               int64_t* nprobes, double* beta_x, int32_t* exit_reason,
                               double* evals, float* evecs, float* psi, void* ws, size_t ws_bytes,
                               void* stream);

/* ---- diagnostics: kernel timing with HIP events ----
 * When enabled, every launch of the fused product kernel (FD_KERNEL_PRODUCT)
 * and of the row-sum kernel of the normalisation passes (FD_KERNEL_ROWSUM) is
 * bracketed by two HIP events recorded on the launch stream (at most 65536
 * brackets per kind are kept; later launches are not timed).
 * fd_profile_read waits for the recorded events, returns the summed kernel time
 * in milliseconds (host) and the number of timed launches (host), and clears
 * the record of that kind. */
typedef enum fd_kernel_kind { FD_KERNEL_PRODUCT = 0, FD_KERNEL_ROWSUM = 1 } fd_kernel_kind;
void fd_profile_enable(int32_t on);
fd_status fd_profile_read(fd_kernel_kind kind, double* total_ms, int64_t* launches);

/* Thread-local message describing the last non-OK status ("" if none). */
const char* fd_last_error(void);

/* Static name of a status code. */
const char* fd_status_string(fd_status s);

#ifdef __cplusplus
}
#endif

#endif /* FLASHDIFF_H */
