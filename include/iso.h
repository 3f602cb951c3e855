/*
 * iso.h -- C ABI of libiso.so: the element-wise merge/update hot path of
 * ISO ("An RLVR-Native Optimization Stack") and the data-free merges it is
 * compared against, as MI355X (gfx950) HIP kernels.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - A call processes a table of n_t 2-D weight tensors (iso_tensor, host
 *    memory, read before the call returns).  Each tensor has a base W_0
 *    (theta_0 restricted to that matrix), K expert deltas tau_i = theta_i -
 *    theta_0 of the same shape (App. F), row-major and contiguous, and
 *    rows*cols = N elements.  1 <= K <= ISO_MAX_K.
 *  - Storage types: ISO_F32 (IEEE binary32) or ISO_BF16 (bfloat16 bits).  One
 *    call uses one storage type for base, deltas and the weight output.
 *  - All data pointers are device memory owned by the caller; every one must
 *    be 16-byte aligned (ISO_ERR_ALIGNMENT otherwise), except the binary64
 *    arrays of iso_frame, iso_spectral_diagnostics, iso_spectral_error and iso_transport_ratios
 *    (8-byte) and the gradient and weight of iso_frame (4-byte).  N need not
 *    be a multiple of anything.
 *  - ws / ws_bytes: caller-allocated device workspace of at least
 *    iso_workspace_size(op, ...) bytes, 256-byte aligned, that must stay
 *    alive until the stream work has finished.  Its contents on entry do not
 *    matter.  The library allocates no device memory.
 *  - stream: a hipStream_t (NULL = the default stream).  Work is queued on
 *    it.  The streaming operations (TopKMask, sign election, merges, APPLY
 *    and FUSED updates) are asynchronous.  The binary64 dense operations
 *    (SPECTRAL, ORTHO, TSV, the diagnostics, the optimizer steps) read
 *    convergence flags on the host between blocks of iterations, so they
 *    synchronise the stream during the call.  Some of their independent
 *    pieces (groups of Jacobi jobs, per-matrix steps) run on streams the
 *    library creates once per device (default priority, kept until the
 *    process ends), forked from `stream` and joined back into it before the
 *    call returns: the call stays ordered on `stream` like any other work.
 *    Concurrent calls on one device share those streams (each keeps its own
 *    dependencies).
 *  - Errors: argument, shape, alignment and workspace-size errors are found
 *    on the host before anything is queued and returned directly.  A
 *    non-finite base or delta value found by a kernel sets a status word in
 *    the workspace; iso_read_device_status returns ISO_ERR_NONFINITE then (the
 *    outputs of such a call are unspecified).  HIP launch errors are
 *    returned as ISO_ERR_HIP.  Nothing throws across the ABI.
 *  - Results are deterministic.  Those of the streaming operations
 *    (TopKMask, sign election, merges, APPLY and FUSED updates) are also
 *    bit-identical however the tensors are grouped into calls and whichever
 *    route (single read or two passes) a call takes.  The binary64 dense
 *    operations (SPECTRAL, TSV, the diagnostics, the optimizer steps) are
 *    bit-identical across runs of the same call; grouping other matrices into
 *    the same call can change where an SVD starts (the warm start of the
 *    experts from the base's factor) and so the last bits of its result.
 *
 * Arithmetic (readings of the paper, which fixes no precision for these
 * operators): every merged coordinate is formed in binary64 -- sums start
 * at +0.0 and add the terms in expert order, means divide that sum by the
 * count, then u = lambda*t and v = w0 + u -- and v is rounded ONCE to the
 * storage type (round to nearest even): the bf16 output is the correct
 * rounding of v, never a double rounding through binary32.  The sign used by
 * the TIES election is the sign of the exact real sum.
 *
 * Entry points: TopKMask (iso_topk_mask, joint over tensor groups), sign
 * election (iso_sign_elect), TIES / TA / RAM merges (iso_merge), the update
 * theta_0 + lambda tau and ISO-Merger (iso_update), TSV (iso_blockdiag_project,
 * iso_blockdiag_project_factors), the ISO-AdamW and ISO-Muon steps
 * (iso_optimizer_step, iso_optimizer_step_muon) and
 * the spectral diagnostics of Sec. 3 (iso_spectral_diagnostics,
 * iso_spectrum_interpolate, iso_transport_ratios) and the mean squared
 * spectral error of App. G (iso_spectral_error).
 */
#ifndef ISO_H
#define ISO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ISO_MAX_K 8

typedef enum iso_status {
  ISO_OK = 0,
  ISO_ERR_INVALID_ARG = 1,
  ISO_ERR_ALIGNMENT = 2,
  ISO_ERR_WORKSPACE = 3,
  ISO_ERR_NONFINITE = 4,
  ISO_ERR_HIP = 5,
  ISO_ERR_UNSUPPORTED = 6,
  ISO_ERR_INTERNAL = 7     /* a kernel met counts that cannot occur; outputs invalid */
} iso_status;

/* The enumerations name the values of plain int parameters and fields: the library checks
 * every such value and answers ISO_ERR_INVALID_ARG to one outside its enumeration. */
typedef enum iso_dtype { ISO_F32 = 0, ISO_BF16 = 1 } iso_dtype;

/* App. F: Task Arithmetic, TIES-Merging, RAM. */
typedef enum iso_merge_mode { ISO_MERGE_TA = 0, ISO_MERGE_TIES = 1, ISO_MERGE_RAM = 2 } iso_merge_mode;

typedef enum iso_update_mode {
  ISO_UPDATE_APPLY = 0,    /* out = W_0 + lambda * tau_in                                   */
  ISO_UPDATE_FUSED = 1,    /* out = W_0 + merged update, elect + merge + apply in one pass  */
  ISO_UPDATE_SPECTRAL = 2, /* out = W_* of ISO-Merger (Algorithm 1)                          */
  ISO_UPDATE_ORTHO = 3     /* out = W_OM of OrthoMerge-G-TIES (App. F)                       */
} iso_update_mode;

/* Operation codes for iso_workspace_size. */
typedef enum iso_op {
  ISO_OP_TOPK = 0,
  ISO_OP_SIGN = 1,
  ISO_OP_MERGE = 2,
  ISO_OP_UPDATE_APPLY = 3,
  ISO_OP_UPDATE_FUSED = 4,     /* FUSED with caller descriptors, or TA / RAM                    */
  ISO_OP_UPDATE_FUSED_SELECT = 5, /* FUSED TIES that selects inside the call (desc == NULL)     */
  ISO_OP_UPDATE_SPECTRAL = 6,
  ISO_OP_BLOCKDIAG = 7,
  ISO_OP_UPDATE_ORTHO = 8
} iso_op;

/* One weight tensor of the table.  Which pointers are read depends on the call. */
typedef struct iso_tensor {
  const void* base;                /* W_0, N elements                                           */
  const void* deltas[ISO_MAX_K];   /* tau_1..tau_K, N elements each (entries >= K ignored)      */
  void* out;                       /* merged weights, N elements of the storage type            */
  int64_t rows, cols;              /* N = rows * cols, N >= 0                                    */
  int64_t k;                       /* TopKMask count per delta, 0 <= k <= N (TIES only)          */
  int32_t select_group;            /* 0: selected alone; > 0: selected jointly with the tensors   */
                                   /* of the same id (see iso_topk_mask)                          */
} iso_tensor;

/*
 * TopKMask of one delta (App. F, TIES "Trim": m_i = TopKMask(|tau_i|, rho)),
 * in threshold form.  key(x) is the storage bit pattern of |x| (bf16: bits &
 * 0x7FFF, fp32: bits & 0x7FFFFFFF), which orders like |x|.  Entry p (flat,
 * row-major) is kept iff key_p > t_key, or key_p == t_key and p < tie_cutoff:
 * exactly k entries, the k largest magnitudes, ties at the threshold going to
 * the lower flat index.  n_above = #{key > t_key}, tie_quota = k - n_above.
 * tie_cutoff is N when every entry with key == t_key is kept, else one past
 * the flat index of the tie_quota-th such entry (so the descriptor is unique).
 * key_max is the largest key in the delta.  k == 0 gives t_key = 0xFFFFFFFF,
 * n_above = tie_quota = tie_cutoff = 0.
 *
 * Joint selection (the paper's TopKMask of a whole-model delta tau_i, App. F):
 * the tensors of one select_group > 0 are selected together, per delta, as
 * if their deltas were concatenated in table order: the K_g largest keys of
 * the concatenation, ties at the threshold going to the earlier tensor and
 * then the lower flat index, with K_g the sum of the members' k (put the
 * whole count on one member or spread it).  The descriptors stay per tensor
 * and per delta, each describing that tensor's part of the joint mask (its
 * n_above + tie_quota is its share of K_g).  bf16 only (ISO_ERR_UNSUPPORTED
 * for an fp32 call with a group); calls with groups take the two-pass path.
 */
typedef struct iso_select_desc {
  uint32_t t_key;
  uint32_t key_max;
  int64_t n_above;
  int64_t tie_quota;
  int64_t tie_cutoff;
} iso_select_desc;

/*
 * Bytes of workspace the given operation needs for this table (0 on bad
 * arguments).  ISO_OP_BLOCKDIAG also needs the rank: use iso_workspace_size_tsv.
 */
size_t iso_workspace_size(int op, const iso_tensor* t, int n_t, int K, int dt);

/*
 * iso_topk_mask -- TopKMask of every delta of every tensor (App. F, TIES
 * "Trim"), k = t[j].k.  Writes desc[j*K + i] (device memory, n_t*K entries)
 * for delta i of tensor j.  If mask_bits is not NULL it is a host array of
 * n_t*K device pointers; pointer j*K+i receives the mask as ceil(N/32)
 * uint32 words, bit (p % 32) of word p/32 set iff entry p is kept.  Exact
 * radix selection over the magnitude keys; the result is unique.
 */
iso_status iso_topk_mask(const iso_tensor* t, int n_t, int K, int dt, iso_select_desc* desc,
                         uint32_t* const* mask_bits, void* ws, size_t ws_bytes, void* stream);

/*
 * iso_sign_elect -- gamma^p = sign(sum_i tilde tau_i^p) (App. F, TIES "Elect
 * Sign"), tilde tau_i = m_i (.) tau_i with m_i from desc (device, n_t*K
 * entries from iso_topk_mask), or tilde tau_i = tau_i when desc is NULL.
 * The sign is that of the exact real sum.  sign_out is a host array of n_t
 * device pointers; tensor j receives N int8 values in {-1, 0, +1}.
 */
iso_status iso_sign_elect(const iso_tensor* t, int n_t, int K, int dt, const iso_select_desc* desc,
                          int8_t* const* sign_out, void* ws, size_t ws_bytes, void* stream);

/*
 * iso_merge -- the merged task vector tau_merge (App. F) as binary32:
 *   ISO_MERGE_TA:   lambda * sum_i tau_i                                   (Task Arithmetic)
 *   ISO_MERGE_TIES: lambda * mean over A_p = {i: tilde tau_i != 0,
 *                   sign(tilde tau_i) = gamma^p}, 0 where A_p is empty       (TIES disjoint mean)
 *   ISO_MERGE_RAM:  lambda * mean over A_p = {i: |tau_i| > eps_act}, 0 if
 *                   empty (the paper's RAM has lambda = 1)                  (RAM)
 * desc is required for TIES and ignored otherwise.  tau_out is a host array
 * of n_t device pointers to N floats: each is the binary64 u = lambda*t
 * rounded once to binary32.
 */
iso_status iso_merge(const iso_tensor* t, int n_t, int K, int dt, int mode,
                     const iso_select_desc* desc, double lambda, double eps_act, float* const* tau_out, void* ws,
                     size_t ws_bytes, void* stream);

typedef struct iso_update_args {
  int mode;                         /* an iso_update_mode                                           */
  int merge;                        /* FUSED: which merge, an iso_merge_mode                      */
  double lambda;                    /* APPLY, FUSED: scale of the merged update (TIES: 1.0)         */
  double eps_act;                   /* FUSED RAM: activity threshold (paper: 1e-5), strict >        */
  const iso_select_desc* desc;      /* FUSED TIES: device descriptors, or NULL to select inside     */
  const float* const* tau_in;       /* APPLY: host array of n_t device pointers, N floats each      */
  int8_t* const* sign_out;          /* FUSED TIES: optional host array of n_t device int8 pointers  */
  double rho_keep;                  /* SPECTRAL: keep ratio (paper 0.9)                             */
  double ridge;                     /* SPECTRAL: lambda_ridge (paper 1e-12)                         */
  double c_min, c_max;              /* SPECTRAL: clip range (paper [0, 1.5])                        */
  double* coef_out;                 /* SPECTRAL: optional device array of n_t*K coefficients c*     */
} iso_update_args;

/*
 * iso_update -- writes t[j].out.
 *  APPLY:    out = round(W_0 + lambda * tau_in)  (theta_merge = theta_0 + tau_merge, App. F).
 *  FUSED:    the merge of iso_merge followed by out = round(W_0 + u) in one
 *            pass that reads each delta and the base once (App. F TIES Trim /
 *            Elect / Merge and theta_0 + lambda tau_TIES; TA; RAM).  With TIES
 *            and desc == NULL the TopKMask selection runs inside the call; for
 *            bf16 (n_t <= 65535) it then reads each delta and the base only
 *            once as well: a sampled key histogram brackets each threshold,
 *            coordinates with a key inside the bracket are logged and fixed up
 *            once the exact threshold is known.  A tensor whose threshold the
 *            bracket misses takes the two-pass path on the device; the result
 *            is the same (iso_read_fallback_count reports how many did).
 *  SPECTRAL: ISO-Merger, Sec. 4.2 / App. E / Algorithm 1, per matrix, in
 *            binary64: SVDs of W_0 and W_i = W_0 + tau_i, joint sign
 *            canonicalisation, tangent projection, D_keep, effect proxies and
 *            their Gram matrix, ridge solve and clip, aggregate projection,
 *            polar retraction, W_* = U_* Sigma_0 V_*^T (rounded once).
 *            Deltas are the raw expert deltas (no TopKMask).  Supported for
 *            min(rows, cols) <= ISO_SPECTRAL_MAX_DIM (the long side is bounded
 *            only by rows * cols < 2^32 and the workspace: binary64 copies of
 *            about 4K + 7 matrices of the tensor's size per call batch).
 *  ORTHO:    OrthoMerge-G-TIES, App. F, per matrix, the geometry-aware
 *            baseline: one-sided Procrustes rotations R_i of the input space
 *            (W_0 R ~ W_i), inverse Cayley maps, magnitude-corrected mean of the
 *            skew matrices, forward Cayley map, W_rot = W_0 R; the residuals
 *            W_i - W_0 R_i (binary32) merged by TIES with the tensor's k as the
 *            TopKMask count (the paper's baseline keeps 20%) and lambda;
 *            out = W_rot + u, u the merged residual update in binary32, rounded
 *            once.  Rotations in binary64 (Jacobi SVDs; the Cayley maps through
 *            symmetric positive definite inverses).  Needs rows >= cols (the
 *            Procrustes rotation of a wide W_0 is not unique) and cols <=
 *            ISO_SPECTRAL_MAX_DIM, else ISO_ERR_UNSUPPORTED; a singular
 *            W_0^T W_i or a rotation with the eigenvalue -1 sets the device
 *            status (ISO_ERR_INTERNAL).  Workspace: ISO_OP_UPDATE_ORTHO.
 */
iso_status iso_update(const iso_tensor* t, int n_t, int K, int dt, const iso_update_args* a, void* ws,
                      size_t ws_bytes, void* stream);

#define ISO_SPECTRAL_MAX_DIM 16384

/*
 * iso_update without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, modes and results as iso_update;
 * the workspace is a fixed block of ISO_NOALLOC_SCRATCH_BYTES of static device
 * memory per GPU, which the library holds until the process ends.  The call
 * allocates nothing.  A call whose workspace (iso_workspace_size of its mode)
 * exceeds the block is rejected with ISO_ERR_UNSUPPORTED before anything is
 * queued; 64 MiB covers, e.g., a fused TopKMask + TIES update of one tensor of
 * about 6M bf16 entries with K = 4.
 * scratch_out (nullable) receives the device address of the current device's
 * block: pass it as the workspace of iso_read_device_status and
 * iso_read_fallback_count after the call.  Every call on one GPU shares that
 * GPU's block, which keeps the last call's contents: calls that overlap on one
 * GPU (other streams or threads) race and must be serialised by the caller.
 * Profiling events (iso_profile_begin) are not recorded by this entry point.
 */
#define ISO_NOALLOC_SCRATCH_BYTES (64ull << 20)

iso_status iso_update_noalloc(const iso_tensor* t, int n_t, int K, int dt, const iso_update_args* a,
                              void** scratch_out, void* stream);

/*
 * Spectral drift diagnostics (Sec. 3), per tensor, in binary64: base = W_0,
 * deltas[0] = Delta W (W_1 = W_0 + Delta W).  out is a device array of 3 n_t
 * doubles, per tensor {delta_Sigma, rho_Sigma, kappa_spec}:
 *   delta_Sigma = |sigma(W_1) - sigma(W_0)|_2 / |W_0|_F,
 *   rho_Sigma   = |sigma(W_1) - sigma(W_0)|_2 / |Delta W|_F,
 *   kappa_spec  = (rows cols / q) |diag(U_0^T Delta W V_0)|_2^2 / |Delta W|_F^2.
 * Workspace: iso_workspace_size(ISO_OP_UPDATE_SPECTRAL, t, n_t, 1, dt); the
 * size limit of ISO-Merger (min(rows, cols) <= ISO_SPECTRAL_MAX_DIM).
 */
iso_status iso_spectral_diagnostics(const iso_tensor* t, int n_t, int dt, double* out, void* ws,
                                    size_t ws_bytes, void* stream);

/*
 * Mean squared spectral error (App. G, the precision study of the SVD behind the
 * polar retraction), per tensor, in binary64:
 *   eps_sigma = (1/q) |sigma(W_rec) - sigma(W_0)|_2^2,  q = min(rows, cols),
 * with W_0 = base and
 *   self_recon = 0: W_rec = deltas[0], a whole matrix of the same shape and
 *                   storage type (not a difference);
 *   self_recon = 1: W_rec = U Sigma V^T formed in binary64 from the library's
 *                   own SVD of W_0 (deltas are not read), the reconstruction
 *                   the appendix measures for each SVD configuration.
 * Singular values come from the binary64 one-sided Jacobi SVD of ISO-Merger.
 * out is a device array of n_t doubles (8-byte aligned); tensors with no
 * elements are skipped.  ISO_ERR_INVALID_ARG for self_recon outside {0, 1}.
 * Same workspace and size limits as iso_spectral_diagnostics.
 */
iso_status iso_spectral_error(const iso_tensor* t, int n_t, int dt, int self_recon, double* out, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * Spectrum interpolation (Sec. 3): out = U_RL [(1 - alpha) Sigma_0 + alpha
 * Sigma_RL] V_RL^T for W_RL = base + deltas[0] and Sigma_0 the spectrum of base
 * (alpha = 0 restores the base spectrum on the trained frames), rounded once.
 * Same workspace and limits as iso_spectral_diagnostics.
 */
iso_status iso_spectrum_interpolate(const iso_tensor* t, int n_t, int dt, double alpha, void* ws,
                                    size_t ws_bytes, void* stream);

/*
 * Unexplained-update ratios (Sec. 3, Prop. 3.1), per tensor, in binary64: the
 * transition from the incoming checkpoint W_j = base to the learned endpoint
 * W_i = base + deltas[0], both truncated to their top-r SVD with
 * r = max(1, floor(f q)), q = min(rows, cols), for each of the n_frac rank
 * fractions f = rank_frac[0 .. n_frac-1] (a host array, 0 < f <= 1,
 * 1 <= n_frac <= ISO_MAX_RANK_FRACS; the paper's main text takes 0.9, its
 * rank-sensitivity study 0.2, 0.4, 0.6, 0.8 and 0.9).  With
 * P_j = U_j^(r) U_j^(r)T and Q_j = V_j^(r) V_j^(r)T the reconstructions are
 * W_mix = P_j W_i^(r) Q_j, W_L = P_j W_i^(r), W_R = W_i^(r) Q_j and
 * W_iso = U_i^(r) Sigma_j^(r) V_i^(r)T, and
 * u_h = |W_i^(r) - W_h|_F / |W_i^(r) - W_j^(r)|_F (u_iso in its closed form
 * |sigma_i^(r) - sigma_j^(r)|_2 / |W_i^(r) - W_j^(r)|_F).  The SVDs are taken
 * once per tensor.  out is a device array of 5 n_frac n_t doubles: tensor j,
 * fraction f at out[5 (j n_frac + f) ...] = {u_mix, u_L, u_R, u_iso, gap},
 * where gap = min over both endpoints of sigma_r - sigma_{r+1}
 * (sigma_{q+1} := 0): the transition is admissible at that rank (its top-r
 * projectors well defined) only when gap > 0, which the caller checks; the
 * ratios are NaN when W_i^(r) = W_j^(r).  Tensors with no elements are
 * skipped (their entries of out are not written).  Workspace and size limits
 * of iso_spectral_diagnostics; ISO_ERR_INVALID_ARG for a fraction outside
 * (0, 1] or n_frac outside [1, ISO_MAX_RANK_FRACS].
 */
#define ISO_MAX_RANK_FRACS 16

iso_status iso_transport_ratios(const iso_tensor* t, int n_t, int dt, const double* rank_frac, int n_frac,
                                double* out, void* ws, size_t ws_bytes, void* stream);

/*
 * ISO-Optimizer step with AdamW as the base rule (ISO-AdamW, Sec. 4.3): one
 * weight matrix W = U Sigma_0 V^T is trained through its frame variables U
 * (rows x rank) and V (cols x rank) with Sigma_0 fixed.  Per frame, in binary64:
 *   G_U = G_W V Sigma_0,  G_V = G_W^T U Sigma_0            (factor gradients)
 *   AdamW on U with (m_u, v_u) and on V with (m_v, v_v):
 *     m <- b1 m + (1 - b1) g,  v <- b2 v + (1 - b2) g^2,
 *     x <- x - lr * ((m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps) + wd x)
 *   U <- polar(U), V <- polar(V),  w_out <- U Sigma_0 V^T (rounded once).
 * U, V, the moments and sigma are device binary64 arrays owned by the caller,
 * column-major (entry (i, k) of U at u[i + k * rows]); U, V and the moments
 * are updated in place.  grad (G_W) and w_out are rows x cols row-major in the
 * storage type.  polar(X) = X (X^T X)^{-1/2} (full column rank), computed as
 * for ISO-Merger.  rank <= min(rows, cols) <= ISO_SPECTRAL_MAX_DIM.
 */
typedef struct iso_frame {
  double* u;            /* rows x rank */
  double* v;            /* cols x rank */
  const double* sigma;  /* rank */
  double* m_u;          /* AdamW: first and second moments of U and of V; */
                        /* Muon: m_u, m_v are the momentum buffers, v_u, v_v unused */
  double* v_u;
  double* m_v;
  double* v_v;
  const void* grad;     /* G_W */
  void* w_out;          /* W+ */
  int64_t rows, cols, rank;
} iso_frame;

typedef struct iso_adamw {
  double lr, beta1, beta2, eps, weight_decay;
  int64_t step;         /* t >= 1: the step being taken (bias corrections 1 - beta^t) */
} iso_adamw;

size_t iso_workspace_size_optimizer(const iso_frame* f, int n_f);
iso_status iso_optimizer_step(const iso_frame* f, int n_f, int dt, const iso_adamw* opt, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * ISO-Optimizer step with Muon as the base rule (ISO-Muon, Sec. 4.3; the
 * paper names the rule without restating it, this is its usual form): the
 * same frames, factor gradients, retraction and output as iso_optimizer_step,
 * with Muon on U (momentum buffer m_u) and on V (momentum buffer m_v):
 *   b <- mu b + g,  d = g + mu b (nesterov != 0) or d = b,  o = polar(d),
 *   x <- x - lr * (sqrt(max(1, rows_x / rank)) o + wd x)
 * where rows_x is rows for U and cols for V.  Muon itself approximates
 * polar(d) by a few quintic Newton-Schulz steps; here o is the polar factor,
 * computed as for the retraction.  v_u and v_v are not used (they may be
 * NULL).  The zero direction (a zero gradient on a zero buffer) takes
 * o = 0, so x only decays; so does a d whose Gram d^T d is exactly zero in
 * binary64 (entries below ~1e-154).  Any other d needs full column rank:
 * otherwise it has no unique polar factor, the iteration does not converge
 * within 48 steps and iso_read_device_status reports ISO_ERR_INTERNAL (a
 * full-rank d converges within the cap up to condition numbers near 1e10:
 * about 20 steps up to 1e5, 35 at 1e8).
 * Workspace: iso_workspace_size_optimizer.
 */
typedef struct iso_muon {
  double lr, momentum, weight_decay;
  int32_t nesterov;
} iso_muon;

iso_status iso_optimizer_step_muon(const iso_frame* f, int n_f, int dt, const iso_muon* opt, void* ws,
                                   size_t ws_bytes, void* stream);

/*
 * iso_blockdiag_project -- TSV-Merge (App. F): each delta is truncated to its
 * top-`rank` singular triplets, the left and right singular vectors are
 * concatenated (U = [U_1 | ... | U_K], V likewise, Sigma = blockdiag of the
 * Sigma_i), U and V are orthogonalised in the Procrustes form (U_perp = P Q^T
 * for U = P D Q^T), and out = round(W_0 + alpha * U_perp Sigma V_perp^T).
 * K*rank <= min(rows, cols).  If delta_hat is not NULL it is a host array of
 * n_t device pointers receiving U_perp Sigma V_perp^T as N floats.
 */
iso_status iso_blockdiag_project(const iso_tensor* t, int n_t, int K, int dt, int rank, double alpha,
                                 float* const* delta_hat, void* ws, size_t ws_bytes, void* stream);

size_t iso_workspace_size_tsv(const iso_tensor* t, int n_t, int K, int dt, int rank);

/* Truncated factors of one delta (App. F, TSV step 1): Delta_i ~ U_i diag(s_i) V_i^T.
 * Device memory, binary64, row-major: u is rows x rank, v is cols x rank, s has rank values. */
typedef struct iso_factors {
  const double* u;
  const double* s;
  const double* v;
} iso_factors;

/*
 * iso_blockdiag_project_factors -- the same projection (concatenation, Procrustes
 * orthogonalisation, reconstruction and update) from given truncated factors
 * instead of the library's own truncated SVD: factors[j*K + i] belong to delta i
 * of tensor j (host array of device pointers).  For callers that already hold
 * the factors, and so that the steps after the SVD can be checked on their own.
 * The deltas of the table are not read; base and out are.  Same workspace as
 * iso_blockdiag_project (iso_workspace_size_tsv) and the same errors.
 */
iso_status iso_blockdiag_project_factors(const iso_tensor* t, int n_t, int K, int dt, int rank, double alpha,
                                         const iso_factors* factors, float* const* delta_hat, void* ws,
                                         size_t ws_bytes, void* stream);

/* round(n * num / den), halves rounded up, in exact integer arithmetic; -1 on bad arguments. */
int64_t iso_k_from_density(int64_t n, int64_t num, int64_t den);

/* Synchronises `stream`, then reports what the kernels of the last call on `ws` found. */
iso_status iso_read_device_status(const void* ws, void* stream);

/* Synchronises `stream`, then stores in *count the number of tensors that the last
 * single-read fused TIES call on `ws` (iso_update, FUSED, TIES, desc NULL, bf16) sent to
 * the exact two-pass path; 0 after any other call.  A performance diagnostic only: the
 * outputs do not depend on it. */
iso_status iso_read_fallback_count(const void* ws, void* stream, int32_t* count);

/* Benchmark timing.  Between iso_profile_begin and iso_profile_end, every iso_update
 * FUSED call records a pair of HIP events on its stream around its main streaming kernel
 * (the single-read pass of the bf16 TIES path with inner selection, else the merge
 * kernel), and iso_optimizer_step / iso_optimizer_step_muon record a pair around each of
 * their Newton-Schulz polar iterations (the retraction; Muon's directions too).
 * iso_profile_end waits for those events and returns the summed elapsed time in
 * milliseconds and the number of regions timed; the library keeps its events for reuse.
 * Calls on several host threads at once are timed too, in no particular order.
 * iso_profile_flops returns the binary64 flops the timed polar iterations performed since
 * iso_profile_begin: per job (frame side of rows x rank, m x q) and step taken, 2 m q^2 for
 * the Gram X^T X (formed whole) and 2 m q^2 for the product X T (0 for the merge paths). */
iso_status iso_profile_begin(void);
iso_status iso_profile_end(double* total_ms, int32_t* launches);
iso_status iso_profile_flops(double* flops);

const char* iso_status_string(int s);

#ifdef __cplusplus
}
#endif

#endif /* ISO_H */
