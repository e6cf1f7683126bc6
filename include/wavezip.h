/*
 * wavezip.h -- C ABI of the WaveZip token-condensation pass on AMD Instinct
 * MI355X (gfx950).
 *
 * The pass implements the query-conditioned condensation C(X, Q) -> Z~ of
 * Sec. 3.1, Eq. (4)-(5): T frames of H x W visual tokens with C channels and a
 * query of Q tokens go in; at most B tokens come out, with per-frame budgets
 * n_t >= 0 that sum to B.  It has four stages, each with its own entry point:
 *
 *   wz_relevance            similarity scores a_{t,n}, frame relevance r_t and
 *                           visual change delta_t (Sec. 3.2.1, Eq. (8));
 *   wz_temporal_budget      gate gamma, frame filter, gated temporal Haar DWT
 *                           and its inverse, and integer budgets
 *                           (Sec. 3.2.2-3.2.3, Eq. (9)-(11); Sec. 3.2.4,
 *                           Eq. (16) with Eq. (5));
 *   wz_spatial_dwt_condense saliency map, per-frame selection and the
 *                           saliency-gated 2-D Haar modulation, compacted in
 *                           temporal order (Eq. (7), Eq. (12)-(15), Eq. (19));
 *   wz_condense             the three stages in sequence;
 *   wz_condense_batch       the same for several videos at once;
 *   wz_condense_queries     the same for several queries over one video.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers: every array argument is a DEVICE pointer owned by the caller.  The
 *   library never allocates, frees or keeps device memory, and keeps no state
 *   between calls.  Arrays are dense, row-major and contiguous.
 * Layouts: X is [T][H][W][C] (channels fastest); query is [Q][C]; both hold
 *   cfg->in_dtype.  A token's flat index is t*H*W + h*W + w (0-based).
 * Alignment: X, query and out_tokens must be 16-byte aligned; float and int32
 *   arrays 4-byte aligned; the workspace 256-byte aligned.
 * Streams: `stream` is a hipStream_t passed as void* (NULL = the default
 *   stream).  All work is enqueued asynchronously on it; nothing is copied
 *   back to the host.  Calls on distinct buffers may run concurrently.
 * Errors: the returned status covers argument validation and kernel-launch
 *   errors only.  When validation fails nothing is enqueued.  Device-side
 *   errors surface on the stream like any HIP error.
 * Determinism: for fixed inputs every output is bitwise reproducible (all
 *   reductions run in a fixed order; no floating-point atomics).
 * Readings of the paper used throughout: with several query tokens a score is
 *   the maximum over query tokens of the cosine; a cosine involving a zero
 *   vector is 0; min-max normalisations of an all-equal input give 0; frame 0
 *   is always retained; odd lengths are extended by repeating the last sample
 *   before each Haar step; Eq. (16)'s rounding is a capped largest-remainder
 *   apportionment (ties to the smaller frame index); the interpolation of
 *   Eq. (17) is replaced by keeping each frame's n_t most salient tokens (ties
 *   to the smaller index) in raster order.
 */
#ifndef WAVEZIP_H
#define WAVEZIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WZ_OK = 0,
  WZ_ERR_NULL = 1,       /* a required pointer is NULL                        */
  WZ_ERR_ALIGN = 2,      /* a pointer violates its alignment                  */
  WZ_ERR_SHAPE = 3,      /* a dimension is out of the supported range         */
  WZ_ERR_DTYPE = 4,      /* unknown in_dtype / out_dtype                      */
  WZ_ERR_PARAM = 5,      /* levels, lambda or tau out of range                */
  WZ_ERR_BUDGET = 6,     /* B < 0 or B > T*H*W                                */
  WZ_ERR_WORKSPACE = 7,  /* workspace smaller than wz_workspace_bytes()       */
  WZ_ERR_DEVICE = 8,     /* a HIP call or kernel launch failed                */
  WZ_ERR_SCRATCH = 9     /* wz_condense_noalloc: the problem needs more than
                            wz_noalloc_scratch_bytes() of scratch             */
} wz_status;

typedef enum { WZ_F32 = 0, WZ_BF16 = 1 } wz_dtype;

/* Wavelet basis of the temporal allocator (Eq. (9)-(11)) or of the spatial
 * modulator (Eq. (12)-(15)).  WZ_HAAR is the orthonormal Haar transform the
 * equations are written with; WZ_DB4 (the paper's spatial default, Sec. 4.1)
 * and WZ_BIOR44 (its basis ablation, Sec. 4.3) use filter banks of 8 and 10
 * taps: Daubechies' minimum-phase N = 4 filter, and the CDF 9/7 pair of
 * JPEG 2000's irreversible transform.  Conventions for the longer banks: one
 * analysis step on L samples extends them half-sample symmetrically and
 * gives floor((L + F - 1) / 2) coefficients per band, a[k] = sum_j
 * dec_lo[j] x~[2k + 1 - j]; synthesis is cropped back to L; a gate is pooled
 * to a subband's length by adaptive average pooling (output i averages
 * inputs floor(i L / n) .. ceil((i + 1) L / n) - 1).                        */
typedef enum { WZ_HAAR = 0, WZ_DB4 = 1, WZ_BIOR44 = 2 } wz_basis;

/* How a frame's n_t output tokens are formed from its modulated map
 * (Token Assigner, Eq. (17)).                                                 */
typedef enum {
  WZ_SELECT = 0,  /* the n_t tokens of largest score, in raster order (default) */
  WZ_INTERP = 1   /* budget-guided bilinear interpolation Psi: the first n_t
                     cells, in raster order, of an h' x w' grid keeping the
                     frame's aspect ratio (h0 = the integer nearest
                     sqrt(n_t H / W), halves up, within [1, H]; w' = min(W,
                     ceil(n_t / h0)); h' = ceil(n_t / w')), cell (i, j) the
                     bilinear interpolation at the half-pixel centre
                     ((2i+1) H / (2h') - 1/2, (2j+1) W / (2w') - 1/2) with
                     negative coordinates clamped to 0; out_index holds the
                     token nearest that point (halves up)                    */
} wz_assign;

/* Problem description.  Supported ranges (anything else is WZ_ERR_SHAPE /
 * WZ_ERR_PARAM): 1 <= T <= 2048; 1 <= H, W and H*W <= 4096; 1 <= Q <= 1024;
 * 8 <= C <= 65536 with C % 8 == 0; 1 <= levels <= 16; lambda_ finite and
 * >= 0; tau in [0, 2]; assign a wz_assign value; spatial_levels 0, 1 or 2
 * (2 only with WZ_SELECT); temporal_basis and spatial_basis wz_basis values;
 * a spatial_basis other than WZ_HAAR needs WZ_SELECT, spatial_levels <= 1,
 * H, W <= 64 and H*W <= 1024.                                                  */
typedef struct {
  int32_t T, H, W, C, Q;
  int32_t in_dtype;   /* wz_dtype of X and query                               */
  int32_t out_dtype;  /* wz_dtype of out_tokens (WZ_F32 keeps full precision)  */
  int32_t levels;     /* J, temporal Haar levels (the paper uses 1)            */
  int64_t B;          /* global token budget, 0 <= B <= T*H*W                  */
  float lambda_;      /* WSM modulation strength (the paper's default: 1.5)    */
  float tau;          /* frame-filter threshold on delta; 0 keeps every frame  */
  int32_t assign;     /* wz_assign (0, the zero-initialised default: selection) */
  int32_t spatial_levels; /* levels of the spatial Haar modulator: 0 or 1 for
                         the single level of Eq. (12)-(15) (default), 2 for two
                         levels -- the approximation decomposed once more, level
                         2's details gated by lambda times M pooled twice (the
                         multi-level variant of the ablations); selection only */
  int32_t temporal_basis; /* wz_basis of the temporal allocator (0: Haar)   */
  int32_t spatial_basis;  /* wz_basis of the spatial modulator (0: Haar)    */
} wz_config;

/* Bytes of device workspace that wz_relevance and wz_condense need for `cfg`
 * (0 if cfg is invalid): per-unit partial sums of the streaming pass, the
 * intermediate scores and frame values, and budgets; with a db4 / bior4.4
 * spatial basis, bf16 inputs and frames too large for the one-kernel form
 * of stage 3 (about 24 x 24 tokens and up), also each kept token's
 * operator row of the modulator (B rows of 4 * 32*ceil(H*W/32) bytes).
 * Contents on entry are ignored; one call at a time per workspace.          */
size_t wz_workspace_bytes(const wz_config* cfg);

/* Stage 1 -- Cross-Modal Scorer (similarity branch, Sec. 3.2.1) and Visual
 * Change Estimator (Sec. 3.2.2, Eq. (8)).  One pass over X computes
 *   tok_score[t*H*W + n] = a_{t,n} = max_j cos(x_{t,n}, q_j)          [T*H*W]
 *   frame_rel[t]         = r_t = max_j cos(v_t, q_j)                  [T]
 *   frame_delta[t]       = delta_t = clamp(1 - cos(v_t, v_{t-1}), 0, 2),
 *                          delta_0 = 0                                  [T]
 * where v_t is the spatial mean of frame t's tokens.  Accumulation is fp32,
 * the frame-level cosines fp64.  ws: at least wz_workspace_bytes(cfg) bytes
 * of device memory.  Two kernel launches: one pass over X (wz_relevance_pass)
 * writing per-unit partials, then a per-frame step adding them in a fixed
 * order.                                                                     */
wz_status wz_relevance(const wz_config* cfg, const void* X, const void* query,
                       float* tok_score, float* frame_rel, float* frame_delta,
                       void* ws, size_t ws_bytes, void* stream);

/* The pass over X that stage 1 starts with -- the one kernel of the whole
 * pass that reads the frames -- on its own.  It writes the per-token scores
 * a_{t,n} to tok_score [T*H*W] where one workgroup sees every channel of a
 * token (always for bf16 inputs with at most 256 query tokens and for fp32
 * inputs; for bf16 with more query tokens, when the grid has no channel
 * slices), and leaves in ws the per-work-unit partial sums that
 * wz_relevance's per-frame step completes r_t, delta_t (and, with channel
 * slices, a_{t,n}) from.  It
 * lets a caller run or time the pass alone; nothing else reads what it
 * leaves in ws.  Same arguments and checks as wz_relevance.  One kernel
 * launch.                                                                     */
wz_status wz_relevance_pass(const wz_config* cfg, const void* X, const void* query,
                            float* tok_score, void* ws, size_t ws_bytes, void* stream);

/* Stage 2 -- Wavelet Temporal Allocator and budget (gate and frame filter of
 * Sec. 3.2.2; Sec. 3.2.3, Eq. (9)-(11); Sec. 3.2.4, Eq. (16) under Eq. (5)).  From r and delta (as produced by wz_relevance):
 * gamma = min-max(delta) over all T frames; retained set M = {0} U
 * {t : delta_t >= tau}; J-level orthonormal Haar DWT of r over M with every
 * detail level multiplied by gamma pair-averaged to its resolution; inverse
 * DWT -> r~; budgets from w = max(r~, 0) (uniform if all zero), capped at
 * H*W per frame, summing to min(B, |M|*H*W).  Arithmetic is fp64.
 * Outputs: budget[T] (0 for dropped frames); offset[T+1] with offset[0] = 0
 * and offset[t+1] = offset[t] + budget[t] (offset[T] = tokens emitted);
 * rel_rect[T] = r~ for retained frames and 0 for dropped ones (may be NULL). */
wz_status wz_temporal_budget(const wz_config* cfg, const float* frame_rel,
                             const float* frame_delta, int32_t* budget,
                             int32_t* offset, float* rel_rect, void* stream);

/* Stage 3 -- Wavelet Spatial Modulator and Token Assigner (Eq. (7),
 * Eq. (12)-(15), Eq. (19)).  Frame t keeps n_t = offset[t+1] - offset[t]
 * tokens: M_t = min-max(tok_score of frame t); keep the n_t tokens of largest
 * score (ties -> smaller index); for each kept token take its 2x2 Haar block
 * of the grid (last row/column repeated when H or W is odd), compute
 * LL/LH/HL/HH, multiply the three detail bands by g = lambda_ * mean(M over
 * the block), invert, and write the token's reconstructed features to row
 * offset[t] + k of out_tokens ([B][C], cfg->out_dtype), k = the token's rank
 * in raster order among the frame's kept tokens; out_index gets its flat
 * index.  cfg->assign = WZ_INTERP forms the frame's n_t rows by the
 * budget-guided interpolation of the modulated map instead (see wz_assign);
 * cfg->spatial_levels = 2 modulates with two Haar levels.  offset ([T+1], as produced by wz_temporal_budget) must start at 0,
 * be nondecreasing with steps of at most H*W and end at offset[T] <= B; rows
 * from offset[T] on are not written, and no row outside [0, B) is ever
 * written whatever offset holds.  Needs no workspace.  One kernel launch.    */
wz_status wz_spatial_dwt_condense(const wz_config* cfg, const void* X,
                                  const float* tok_score, const int32_t* offset,
                                  void* out_tokens, int32_t* out_index,
                                  void* stream);

/* The whole pass C(X, Q) of Eq. (4)/(6): stage 1, 2 and 3 in sequence on one
 * stream, intermediates kept in `ws`.  Three kernel launches: the pass over
 * X, the per-frame scores, and one kernel that computes the budgets (every
 * workgroup alike) and performs stage 3; for T > 256, a db4 / bior4.4
 * temporal basis, or a db4 / bior4.4 spatial basis with T > 64 the budgets
 * get a launch of their own, and with a db4 / bior4.4
 * spatial basis on large frames (bf16 inputs) stage 3 takes two: the
 * modulator's operator rows of the kept tokens, once per frame, into the
 * workspace, then their product with the frames' channels.  out_tokens [B][C] (cfg->out_dtype) and
 * out_index [B] receive offset[T] rows (= B unless the frame filter leaves
 * fewer than B tokens).  budget [T] and offset [T+1] are optional outputs
 * (NULL: kept in the workspace).                                              */
wz_status wz_condense(const wz_config* cfg, const void* X, const void* query,
                      void* out_tokens, int32_t* out_index, int32_t* budget,
                      int32_t* offset, void* ws, size_t ws_bytes, void* stream);

/* Several videos of one shape condensed in one call: the whole pass of
 * wz_condense for each of `videos` videos (1 <= videos <= 8, else
 * WZ_ERR_SHAPE), every kernel launched once for all of them, so launch and
 * kernel-boundary costs are shared and the videos' work overlaps (a
 * throughput mode for short videos; each video keeps its own query and its
 * own budget B).  Layouts add a leading video index: X [V][T][H][W][C],
 * query [V][Q][C], out_tokens [V][B][C], out_index [V][B] (flat index within
 * the video), budget [V][T] and offset [V][T+1] (optional, NULL: kept in the
 * workspace).  ws: at least videos * wz_workspace_bytes(cfg) bytes, video v
 * using the v-th slice of that size.  Video v's outputs are bitwise those of
 * wz_condense on video v alone.                                             */
wz_status wz_condense_batch(const wz_config* cfg, int32_t videos, const void* X,
                            const void* query, void* out_tokens,
                            int32_t* out_index, int32_t* budget,
                            int32_t* offset, void* ws, size_t ws_bytes,
                            void* stream);

/* Several queries over one video in one call: the whole pass of wz_condense
 * for each of `queries` queries of Q tokens (1 <= queries <= 8, else
 * WZ_ERR_SHAPE) on the same X, each with its own budgets and outputs.  The
 * paper scores every query afresh; here, when the inputs are bf16 and
 * Q <= 32, each pass over X serves a group of up to 64 / Q queries: their
 * tokens are the columns of one relevance contraction, and a_{t,n}, r_t and
 * the selection are taken per query.  Otherwise each query takes its own
 * pass over X (launched together, as in wz_condense_batch).  Layouts:
 * X [T][H][W][C], query [G][Q][C], out_tokens [G][B][C], out_index [G][B],
 * budget [G][T] and offset [G][T+1] (optional, NULL: kept in the
 * workspace).  ws: at least queries * wz_workspace_bytes(cfg) bytes, query g
 * using the g-th slice of that size.  Query g's outputs are bitwise those of
 * wz_condense with query g alone.                                            */
wz_status wz_condense_queries(const wz_config* cfg, int32_t queries,
                              const void* X, const void* query,
                              void* out_tokens, int32_t* out_index,
                              int32_t* budget, int32_t* offset, void* ws,
                              size_t ws_bytes, void* stream);

/* wz_condense without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, outputs and results as wz_condense
 * (bitwise), minus ws / ws_bytes: the intermediates live in a static device
 * array of wz_noalloc_scratch_bytes() = 32 MiB that the library holds on each
 * GPU it runs on until the process ends.  When wz_workspace_bytes(cfg)
 * exceeds that only through the filter-bank operator rows, the modulator
 * keeps them in LDS instead (its one-kernel form; the same results); a
 * problem that does not fit even then returns WZ_ERR_SCRATCH before anything
 * is enqueued.  The call allocates and frees nothing; its first call on a
 * device looks up that device's array (hipGetSymbolAddress) under a lock.
 * Every call on one GPU shares that GPU's array: calls that overlap on one GPU
 * (other streams, other host threads) race and must be serialised by the
 * caller.  Nothing in the array needs clearing between calls (every value is
 * written before it is read in the same call).                              */
wz_status wz_condense_noalloc(const wz_config* cfg, const void* X,
                              const void* query, void* out_tokens,
                              int32_t* out_index, int32_t* budget,
                              int32_t* offset, void* stream);

/* Bytes of the static scratch array behind wz_condense_noalloc (32 MiB).     */
size_t wz_noalloc_scratch_bytes(void);

/* Static, human-readable name of a status code.                               */
const char* wz_status_str(wz_status s);

#ifdef __cplusplus
}
#endif

#endif /* WAVEZIP_H */
