// Internal declarations shared by the gfx950 kernels and the C-ABI layer.
//
// Encoded configurations are arrays of 32-bit "code words" grouped by how the
// per-parameter distance of Sec. 4.1 is evaluated on them:
//   NUM  : one fp32 code u in [0,1] per real/integer/ordinal parameter
//          (term (u - u')^2, weight 1 / l^2);
//   BITS : bit sets whose Hamming distance popc(a ^ b) is the term: one-hot fields of
//          categorical parameters (2 bits differ per changed category, weight
//          1 / (2 l^2)), the pair-order bits [pi_i > pi_j] (i < j) of a Kendall
//          permutation (weight 1 / (l^2 Dmax)), and one-hot item positions of a
//          Hamming permutation (64 bits = 2 words, weight 1 / (2 l^2 Dmax));
//   EQ   : one word compared for equality (categoricals with > 32 levels, naive
//          permutations packed as 4-bit positions), weight 1 / l^2;
//   DOT  : the 8 positions of a Spearman permutation as bytes (2 words); the term is
//          sum (pi_i - pi'_i)^2 = 2 (S2 - pi . pi') with S2 = sum_k k^2 (exact in
//          integers), so the dot product is taken with v_dot4.
// Words are laid out NUM | BITS | EQ | DOT.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstddef>

#include "baco_gp.h"

namespace bgp {

constexpr int kMaxD = 64;
constexpr int kMaxWords = 160;       // code words per configuration
constexpr int kMaxBitsWords = 64;
constexpr int kMaxEqWords = 64;
constexpr int kMaxDot = 16;          // Spearman permutations
constexpr int kMaxN = 4096;          // observations
constexpr int kKChunk = 32;          // K* row stride granularity (contraction k-chunk)
constexpr int kRowTile = 128;        // contraction row tile; M is padded to it
constexpr int kColTile = 128;        // contraction column tile
constexpr int kMaxTiles = 96;        // contraction column tiles (reg + cls)
constexpr int kNB = 32;              // fp64 factorisation block

// One parameter as the encoder sees it (device table, encode order).
struct ParamEnc {
  int32_t kind;      // gp_ptype
  int32_t col;       // index of the caller's raw column
  int32_t word;      // first code word written by this parameter
  int32_t bit;       // CAT: first bit of its one-hot field in `word`, -1 = EQ word
  int32_t levels;    // CAT levels, ORD values, PERM m
  int32_t flags;     // bit 0: log2 transform; bits 8..15: gp_permdist
  int32_t table;     // ORD: offset of its transformed values in the value table
  int32_t num_index; // NUM code index (0..n_num-1), -1 otherwise
  double lo;         // INT/REAL declared range (validity check)
  double hi;
  double t_lo;       // transformed low end
  double den;        // transformed range t_hi - t_lo (0: single value -> code 0)
};

// Word-group counts and the fp64 weights of the distance.
struct Weights64 {
  int32_t n_num, n_bits, n_eq, n_dot;
  int32_t w_bits0, w_eq0, w_dot0, pad;
  double num_w[kMaxD];         // 1 / l^2
  double bits_w[kMaxBitsWords];
  double eq_w[kMaxEqWords];
  double dot_w2[kMaxDot];      // 2 w of a Spearman permutation (term 2 w (S2 - dot))
  int32_t dot_s2[kMaxDot];     // S2 = sum_{k<m} k^2
};

// Per-parameter description used by the term-inspection kernel (space order).
struct TermDesc {
  int32_t kind;   // gp_ptype
  int32_t word;   // first word
  int32_t bit;    // CAT one-hot offset, -1 = EQ
  int32_t m;      // PERM items; CAT levels (one-hot field width)
  int32_t dist;   // gp_permdist
};

// Position of observation i (0..31 within a 32-wide chunk) in a stored K* chunk and in
// the packed B^T: the cross-kernel's MFMA result gives lane group g observations g + 4 v
// of each 16-observation block, and a lane stores its 8 values of a chunk contiguously,
// so observation 16 ob + g + 4 v sits at 8 g + 4 ob + v. (A permutation within each
// chunk, applied alike to both operands of the contraction.)
__host__ __device__ inline int kpos(int i) { return 8 * (i & 3) + 4 * (i >> 4) + ((i >> 2) & 3); }

// Words of a cross-kernel observation record for NB BITS, NE EQ words and ND Spearman
// permutations: alpha (fp64) and |alpha| of 8 observations, then each word of the 8.
__host__ __device__ constexpr int xrec_words(int nb, int ne, int nd) {
  return 24 + 8 * (nb + ne + 2 * nd);
}

// fp32 cross-kernel + candidate-side accumulations.
struct XArgs {
  const uint32_t *cand;  // SoA candidate codes [R][ldc]
  int64_t ldc;
  const double *xa64;    // observation MFMA operands [chunks][2][KS][64]
  const uint32_t *xr;    // observation records [chunks][4][record words]
  int32_t n, lda;
  int32_t n_num, n_bits, n_eq, n_dot;
  int32_t w_bits0, w_eq0, w_dot0;
  int32_t i_chunk;               // observations per split (multiple of 32; >= n if unsplit)
  double num_scale64[kMaxD];     // 1 / l of each numeric code
  float bits_w[kMaxBitsWords];
  float eq_w[kMaxEqWords];
  float dot_w2[kMaxDot];         // 2 w
  int32_t dot_s2[kMaxDot];       // S2 = sum_{k<m} k^2
  float A0, A1, A2;              // 2^kexp (s, s sqrt5, 5 s / 3): Matern-5/2 polynomial,
                                 // scaled so that K* comes out scaled by 2^kexp
  float kinv;                    // 2^-kexp: unscales mu and sens
  uint16_t *Kstar;               // split fp16 K* [rows][2 lda] (layout below)
  double *mu;                    // [rows] sum_i k_i alpha_i  (fp64 accumulation)
  float *sens;                   // [rows] sum_i k_i |alpha_i|
                                 // (split launches: [splits][rows] partial sums)
  int64_t rows;                  // rows to produce (multiple of 64)
  // inspection instantiation only: per pair (j < dbg_count, i < n) the squared
  // distance r2[j][i] and the integer semimetric sum of every BITS, EQ and Spearman
  // word cnt[j][i][w] (w over n_bits + n_eq + n_dot), as the production pass forms them
  float *dbg_r2;
  int32_t *dbg_cnt;
  int64_t dbg_count;
};


// Split fp16 operand layout of the variance contraction. A row of K* (or of the packed
// B^T) is stored per 32-wide k-chunk as 64 halves: the high parts h = fp16(x) of its 32
// values, then the low parts l = fp16(x - h), so that h + l carries about 22 bits of x.
// The fp32 products x y are formed as h_x h_y + h_x l_y + l_x h_y on fp16 MFMA with
// fp32 accumulation (the dropped l_x l_y is 2^-22 relative). Both operands are scaled
// by powers of two first (K* by 2^kexp, column j of B by its own 2^e_j) to keep the low
// parts clear of the fp16 subnormal range; the contraction undoes the scaling of each
// output column with cscale[j] = 2^-(kexp + e_j). A row occupies 4 lda bytes, as an
// fp32 row would.
constexpr int kSplitTop = 14;  // scaled magnitudes lie below 2^(kSplitTop + 1)

struct CTile {
  int32_t bcol;  // first row of the packed B^T for this column tile
  int32_t kend;  // contraction length (multiple of kKChunk)
  int16_t tri0;  // index of the tile's first column within its triangular factor
  int16_t ncol;  // columns of the tile that are not padding (<= kColTile)
  int32_t lin;   // column of the tile (at or past ncol) holding a dense vector whose
                 // product with K* is output as is rather than squared; -1: none
};

struct CArgs {
  const uint16_t *A;    // split K* [rows][2 lda]
  const uint16_t *Bt;   // split packed B^T [ncols][2 lda]
  const float *cscale;  // [ncols] output column unscaling 2^-(kexp + e_j)
  int32_t lda, ntiles, nrowtiles, pad;
  float *part;        // [ntiles][rows]
  float *lin;         // [rows] K* times the linear column (if a tile has one)
  int64_t rows;
  CTile tiles[kMaxTiles];
};

struct EArgs {
  const float *part;
  int64_t rows;
  int64_t M;
  int32_t ntiles, has_cls;
  int32_t n_reg_tiles, pad;            // tiles t >= n_reg_tiles are classifier tiles
  const double *mu64;
  const float *sens;
  const float *fbar;
  const uint8_t *valid;
  const uint8_t *mask;
  float eps_f;
  float sv, cls_sv;
  float fstar;
  float refine_var, refine_sens;  // flag thresholds
  const double *fstar_dev;        // f* on the device (read instead of fstar when set)
  const double *pmu;              // nsplit > 1: the cross-kernel's per-split partial mu and
  const float *psens;             // sens [nsplit][rows], summed here in split order
  int32_t nsplit, pad2;
  float *mu, *sigma, *ei, *p_feas, *acq;
  int32_t *refine_list;
  int32_t *refine_count;
};

struct RArgs {
  const uint32_t *cand;     // SoA codes [R][ldc]
  int64_t ldc;
  const uint32_t *obs;      // AoS unscaled codes [n][R] (model order)
  int32_t R, n_f, cb, ldb;
  const double *B64;        // L_f^-T row-major [n_f][ldb] (upper triangular)
  const double *alpha;      // [n_f]
  const int32_t *list;
  const int32_t *count;
  double sv, fstar;
  const uint8_t *mask;
  float eps_f;
  float *mu, *sigma, *ei, *p_feas, *acq;
  double *part;             // split path: [groups][ceil(n_f / 64)][cb] partial |v|^2
  double *mup;              // split path: [groups][cb] mu
  double *part64;           // block path: [ceil(n_f / 256)][cap] partial |v|^2
  double *mu64;             // block path: [cap] mu
  int64_t cap;              // flagged candidates the block path's buffers hold (>= count)
};
// Up to kRefineSplitGroups groups of cb flagged candidates are recomputed with the
// triangular product split over 64-column ranges (one workgroup per group and range),
// so that a few flagged candidates still spread over many workgroups.
constexpr int kRefineSplitGroups = 16;
constexpr int kRefineColRange = 64;
// More than kRefineBlockMin flagged candidates take the block path: fp64 MFMA over
// groups of kRefineBlockRows candidates and column tiles of kRefineBlockCols.
constexpr int kRefineBlockMin = 4096;
constexpr int kRefineBlockRows = 64;
constexpr int kRefineBlockCols = 256;

// Local search over the acquisition function (search.hip). Configurations in the raw
// column formats as 4-byte words per parameter (REAL 2, INT/ORD/CAT 1, PERM m).
constexpr int kLsMaxStarts = 64;
constexpr int kLsMaxWords = 8 * kMaxD;  // 4-byte words of one raw configuration
struct LSDesc {
  int32_t d, nnb;                 // parameters; neighbours per configuration
  int32_t W, pad;                 // words of one configuration (all parameters)
  uint8_t kind[kMaxD];            // gp_ptype
  uint8_t words[kMaxD];           // 4-byte words per configuration (<= 8)
  uint16_t woff[kMaxD];           // first word of each parameter in the W words
  uint8_t wparam[kLsMaxWords];    // parameter of each of the W words
  uint8_t log2[kMaxD];            // REAL: steps in log2(value)
  uint8_t penc_of[kMaxD];         // index of each parameter's entry in the encode order
  int32_t move0[kMaxD];           // first neighbour index of each parameter
  int32_t lo[kMaxD], hi[kMaxD];   // INT value range, ORD index range
  double t_lo[kMaxD], t_hi[kMaxD];  // REAL: transformed range
};  // passed by value: about 2.7 KB of kernel arguments
struct LSCols {
  uint32_t *col[kMaxD];
};
// Indices (and values) of the k <= kLsMaxStarts largest of acq[0..M) (lower index
// first on ties) into idx / v; pv, pi: parts * k scratch.
hipError_t launch_ls_topk(const float *acq, int64_t M, int k, float *pv, int64_t *pi, int parts,
                          float *v, int64_t *idx, hipStream_t s, const int64_t *map = nullptr);
// (map: the index of element q is map[q] rather than q)
// ub[j] >= the acquisition value of candidate j, from its cross-kernel mean (mu64, sens),
// validity and mask; f* and smax = sqrt(signal variance); *count = 0
hipError_t launch_ls_bound(const double *mu64, const float *sens, const uint8_t *valid,
                           const uint8_t *mask, int64_t M, double fstar, double smax, float *ub,
                           int32_t *count, hipStream_t s);
// the indices with ub >= *tau into list (at most cap of them), their number into *count
hipError_t launch_ls_compact(const float *ub, int64_t M, const float *tau, int64_t *list,
                             int32_t *count, int64_t cap, hipStream_t s);
// configurations idx[0..n) of C into rows 0..n of G, and mask[idx[i]] into mg (if mask)
hipError_t launch_ls_gather_rows(const LSDesc &d, const LSCols &C, const int64_t *idx, int64_t n,
                                 const LSCols &G, const uint8_t *mask, uint8_t *mg, hipStream_t s);
hipError_t launch_ls_gather(const LSDesc &d, const LSCols &C, int64_t M, const int64_t *start,
                            const float *start_v, int k, const LSCols &cur, float *cur_acq,
                            int32_t *active, int32_t *steps, hipStream_t s);
// The scorer's candidate buffers, which a local-search step fills with the codes of the
// neighbours (SoA words [R][rows], rows = k * nnb rounded up to the row tile; padding
// rows repeat the last neighbour).
struct LSEnc {
  const ParamEnc *penc;
  const double *table;
  uint32_t *cand;
  uint8_t *valid;
  int32_t *clear;  // the scorer's counter, set to 0
  int64_t rows;
  int32_t R, pad;
};
// One step of the climb for each of the k starts: if nb_acq is given (the scores of the
// previous step's neighbours), the move to the best of them when that is strictly better;
// then, if gen, the codes, validity and mask of the new neighbours.
hipError_t launch_ls_step(const LSDesc &d, const LSCols &cur, int k, int32_t *active,
                          const float *nb_acq, float *cur_acq, int32_t *steps, int32_t max_steps,
                          bool gen, const LSEnc &e, uint8_t *mask, hipStream_t s);

// Kernel launchers (defined in the .hip files). All enqueue on `s`.
hipError_t launch_encode(const void *const *cols, int32_t d, const ParamEnc *penc,
                         const double *table, int64_t count, int64_t rows_out,
                         const int32_t *rowmap, uint32_t *out, int64_t s_word,
                         int64_t s_row, uint8_t *valid, float *num_out, int32_t n_num,
                         int32_t *clear, hipStream_t s);
// Observation splits of the cross-kernel: 1 when the candidate waves (rows / 64) alone
// fill the chip, else enough splits of the observations (whole 32-chunks each) for about
// 1024 waves. A split launch writes per-split partial sums to XSplit and adds them in
// split order into a.mu / a.sens.
int xkernel_splits(int64_t rows, int n);
struct XSplit {
  int nsplit;
  double *mu;    // [nsplit][rows], only for nsplit > 1
  float *sens;
};
// reduce: sum the per-split partials into a.mu, a.sens (else the consumer sums them)
hipError_t launch_xkernel(const XArgs &a, int variant, const XSplit &sp, hipStream_t s,
                          bool inspect = false, bool reduce = true);
int xkernel_splits(int64_t rows, int n);
int xkernel_variant(int n_num, int n_bits, int n_eq, int n_dot);
// The observation side of the cross-kernel for a variant: MFMA k-steps, padded word
// counts and record width, with the space's natural counts and word offsets.
struct XObsLayout {
  int32_t ks, nb, ne, nd, rw;
  int32_t n_num, n_bits, n_eq, n_dot;
  int32_t w_bits0, w_eq0, w_dot0;
};
XObsLayout xobs_layout(int variant, int n_num, int n_bits, int n_eq, int n_dot, int w_bits0,
                       int w_eq0, int w_dot0);
size_t xobs_a_doubles(int n, int ks);   // size of the MFMA operand array
size_t xobs_r_words(int n, int rw);     // size of the record array
size_t xobs_a_doubles_max(int n);       // the same for the largest variant
size_t xobs_r_words_max(int n);
// Builds both from the observation codes [n][R] (model order), 1 / l of each numeric
// code and alpha (rows < n_f; 0 past them).
hipError_t launch_make_xobs(const uint32_t *codes, int32_t R, int32_t n, const XObsLayout &lay,
                            const double *num_scale, const double *alpha, int32_t n_f,
                            double *xa, uint32_t *xr, hipStream_t s);
hipError_t launch_contract(const CArgs &a, hipStream_t s);
// pwork: float[M] receiving p_feas (the caller's p_feas output or workspace); the
// refinement pass reads it back.
// The value model's half of the epilogue (mu, sigma, EI of the candidates kept in fp32,
// the list of those recomputed in fp64) and the classifier's half (p, acq), which reads
// the EI the first half wrote.
hipError_t launch_epilogue_value(const EArgs &a, hipStream_t s);
hipError_t launch_epilogue_cls(const EArgs &a, float *pwork, hipStream_t s);
// both of the above in one kernel (when they share a stream)
hipError_t launch_epilogue(const EArgs &a, float *pwork, hipStream_t s);
int refine_candidates_per_block(int n_f);
// fp64 recomputation of the flagged candidates: the block path's products (more than
// kRefineBlockMin flagged; needs the value model only; cus: compute units the stream
// can use), then the rest, which writes every output of the flagged candidates (needs
// p in pwork).
hipError_t launch_refine_block(const RArgs &a, const Weights64 &w, int cus, hipStream_t s);
hipError_t launch_refine_rest(const RArgs &a, const Weights64 &w, const float *pwork, int grid,
                              hipStream_t s);
hipError_t launch_argmax(const float *acq, int64_t M, float *pval, int64_t *pidx,
                         int nblocks, int64_t *out, hipStream_t s);
hipError_t launch_terms(const uint32_t *cand, int64_t ldc, const uint32_t *obs, int32_t R,
                        int32_t n, int64_t count, const TermDesc *td, int32_t d,
                        float *terms, hipStream_t s);
// dst[r][c] = (h + l) * inv_scale for the split rows of src (row stride 2 lda halves).
hipError_t launch_gather_rows_split(const uint16_t *src, int32_t lda, float inv_scale, float *dst,
                                    int64_t ld_dst, int64_t rows, int32_t cols, hipStream_t s);

// ------------------------------------------------ hyperparameter fit (hyper.hip)
// A setting theta = (log l_1..log l_d, log s, t), noise variance = floor + e^t.
constexpr int kHypBatch = 64;        // settings per batched evaluation
constexpr int kHypMaxD = kMaxD + 2;  // entries of a setting
constexpr int kHypGradChunk = 32;    // lengthscale gradients accumulated per launch plane
constexpr int kLbfgsMem = 10;        // stored (s, y) pairs
constexpr int kHypGradBlocks = 128;  // pair-range blocks of the gradient contraction
constexpr int kLbfgsMaxHalvings = 30;  // step halvings before a line search gives up

struct HypArgs {
  const double *T;        // [d][nf][nf] per-parameter squared distances / their maxima
  const double *y;        // [nf] targets of the feasible observations
  const double *theta;    // setting b at theta + b * theta_ld
  int64_t theta_ld;
  int32_t d, nf, ld;      // parameters, observations, leading dimension of the matrices
  int64_t sM;             // elements between consecutive settings' matrices
  int64_t sA;             // ... of A (K, the identity rows below it, then K^-1)
  double noise_floor;
  int32_t has_prior;
  double prior_shape, prior_rate, prior_c0;  // c0 = shape log(rate) - lgamma(shape)
  int32_t *info;          // [B] per setting: 0 evaluate, nonzero skip / not a kernel
  const int32_t *active;  // [B] or null: settings to evaluate
};

// T[p][i][j] for the first nf observations (AoS codes, R words each)
hipError_t launch_hyp_terms(const uint32_t *codes, int32_t R, const TermDesc *td, int32_t d,
                            int32_t nf, double *T, hipStream_t s);
// info[b] = !active[b]; K_b = s Matern52(r) + noise I (full nf x nf, leading dim ld) and
// the identity in the nf rows below it (plane stride sA)
hipError_t launch_hyp_gram(const HypArgs &a, int B, double *K, hipStream_t s);
// value[b] (-inf when not a kernel) and alpha_b = K_b^-1 y from L_b and X_b = L_b^-1
// (z: [B][nf] scratch, z_b = X_b y)
hipError_t launch_hyp_value(const HypArgs &a, int B, const double *L, const double *X,
                            double *value, double *alpha, double *z, hipStream_t s);
// grad[b][0..d+1] from Kinv_b = K_b^-1 and alpha_b; part: hyp_grad_part_elems(B, d)
int64_t hyp_grad_part_elems(int B, int d);
hipError_t launch_hyp_grad(const HypArgs &a, int B, const double *Kinv, const double *alpha,
                           double *part, double *grad, int64_t grad_ld, hipStream_t s);
// keep[0..k) = indices of the k largest v[0..S) (NaN as -inf, lower index first on ties),
// x[r] = theta0[keep[r]] (D entries each)
hipError_t launch_hyp_select(const double *v, int32_t S, int32_t k, const double *theta0,
                             int32_t D, int32_t *keep, double *x, hipStream_t s);

struct LbfgsState {
  double *x, *xt, *g, *p;  // [K][D]: iterate, trial point, gradient of F = -objective, direction
  double *S, *Y;           // [K][kLbfgsMem][D] stored pairs (ring)
  double *sy;              // [K][kLbfgsMem] s'y of the stored pairs
  double *F, *t, *slope;   // [K]
  int32_t *status;         // [K] 0 running; 1 gradient tolerance; 2 objective change;
                           //     3 iteration limit; 4 line search failed; 5 start not a kernel
  int32_t *phase, *it, *halv, *npairs, *head;  // [K]
  int32_t *active;         // [K] status == 0 (the evaluator's mask)
};
struct LbfgsParams {
  int32_t D, max_iter;
  double gtol, ftol;
};
// x (already in st.x) becomes the first trial point
hipError_t launch_lbfgs_init(const LbfgsState &st, int K, int32_t D, hipStream_t s);
// value[k] = -F (the objective at the final iterate), iterations and status (may be null)
hipError_t launch_lbfgs_outputs(const LbfgsState &st, int K, double *value, int32_t *iters,
                                int32_t *status, hipStream_t s);
// consume value/grad of the trial points, advance every running start
hipError_t launch_lbfgs_step(const LbfgsState &st, int K, const LbfgsParams &prm,
                             const double *value, const double *grad, int64_t grad_ld,
                             hipStream_t s);

// ------------------------------------------------ Chain-of-Trees (cot.hip)
// Known constraints (Sec. 4.2): each tree of co-dependent INT/ORD/CAT parameters holds
// its feasible partial configurations as sorted bit-packed keys of their value indices
// (level l in a field of bits(dim_l - 1) bits, the first level most significant, so key
// order is the lexicographic order of the leaves); other parameters are free.
constexpr int kCotMaxTrees = kMaxD;
struct CotDesc {
  int32_t d, n_trees, words;      // parameters, trees, random words per configuration
  int32_t pad;
  int32_t kind[kMaxD];            // gp_ptype
  int32_t tree[kMaxD];            // tree of the parameter, -1 free
  int32_t dim[kMaxD];             // values (INT: hi - lo + 1), PERM: m
  int32_t lo[kMaxD];              // INT: lo (raw value = lo + index), else 0
  int32_t shift[kMaxD];           // position of the parameter's field in its tree's key
  uint32_t fmask[kMaxD];          // field mask (2^width - 1)
  double rlo[kMaxD], rhi[kMaxD];  // REAL: declared range
  int32_t tstart[kCotMaxTrees], tcount[kCotMaxTrees];  // tree t: params tparam[tstart..+tcount)
  int32_t tparam[kMaxD];
  int64_t koff[kCotMaxTrees];     // first key of tree t
  int64_t nleaves[kCotMaxTrees];
};
struct CotCols {
  void *col[kMaxD];
};
// keys of tree t's leaves (int32 value indices [n][k]); *bad = lowest leaf index that is
// out of range or not above its predecessor (INT64_MAX if none; must hold INT64_MAX)
hipError_t launch_cot_keys(const CotDesc *dd, int tree, const int32_t *leaves, int64_t n,
                           uint64_t *keys, unsigned long long *bad, hipStream_t s);
hipError_t launch_cot_sample(const CotDesc *dd, const uint64_t *keys, int64_t M, uint64_t seed,
                             uint64_t offset, const CotCols &out, hipStream_t s);
hipError_t launch_cot_member(const CotDesc *dd, const uint64_t *keys, const CotCols &cols,
                             int64_t M, uint8_t *mask, hipStream_t s);

// ------------------------------------------------ random-forest feasibility (forest.hip)
// Hidden constraints (Sec. 4.2): a classification forest of CART trees on bootstrap
// samples of the observations; features are REAL/INT values, ORD/CAT indices and PERM
// positions (one per item), stored as fp64.
constexpr int kForestMaxF = 120;     // features (prediction keeps 64 x F fp64 in LDS)
constexpr int kForestMaxMtry = 16;   // features tried per node (floor(sqrt(F)))
struct ForestDesc {
  int32_t d, F, n, n_trees, max_depth, min_split, mtry, cap;  // cap: nodes per tree (2n)
  uint64_t seed;
  int32_t kind[kMaxD];   // gp_ptype of each parameter
  int32_t fofs[kMaxD];   // first feature of each parameter
  int32_t m[kMaxD];      // PERM items (1 otherwise)
};
struct ForestNode {      // internal: feature >= 0, x_f <= val goes to child `left`, else
  int32_t feature;       // left + 1; leaf: feature = -1, val = feasible fraction
  int32_t left;
  double val;
};
// features [F][ld] (column-major) of `count` configurations given as raw columns
hipError_t launch_forest_features(const ForestDesc *dd, const CotCols &cols, int64_t count,
                                  int64_t ld, double *X, hipStream_t s);
// one workgroup per tree; idx, tmp: [n_trees][n]; nodes [n_trees][cap]; aux [n_trees][cap][3]
hipError_t launch_forest_train(const ForestDesc *dd, int n_trees, const double *X,
                               const uint8_t *y, int32_t *idx, int32_t *tmp, ForestNode *nodes,
                               int32_t *aux, int32_t *n_nodes, hipStream_t s);
// p = mean over trees of the leaf values; acq = ei * p if allowed and p > eps_f else 0
hipError_t launch_forest_predict(const ForestDesc *dd, const ForestDesc &hd, const ForestNode *nodes,
                                 const CotCols &cols, int64_t M, const float *ei,
                                 const uint8_t *mask, float eps_f, float *p, float *acq,
                                 hipStream_t s);

// fp64 linear algebra (linalg.hip)
hipError_t launch_gram(const uint32_t *codes, int32_t R, int32_t n, const Weights64 &w,
                       double sv, double noise, double *K, int32_t ld, hipStream_t s);
// Blocked Cholesky (chol.hip): factor A (destroyed) into L (lower, upper zeroed) and the
// inverses D[k] (kNB x kNB, row-major) of its diagonal blocks; first failing pivot
// (1-based) into *info, which must be 0 on entry. A holds n + n_extra rows: the extra
// rows E (rows n.., columns 0..n-1) are carried along and LE (n_extra x n, leading
// dimension ldle) receives E L^-T. Only the lower triangle of L is written: the upper
// one is cleared first unless clear_upper is false (it is already zero from an earlier
// factorisation into the same L). Kernels return at once when *halt != 0 (halt may be
// null). n_ident = n declares the last n extra rows (starting on a kNB boundary) an
// identity block, whose L_E rows become L^-T: the blocks of L_E below its diagonal
// blocks are never written and must hold zeros.
// first_block_done: L's first diagonal block and D[0] are already there (from
// launch_newton_setup), so the first launch is skipped.
// A batch of independent factorisations of equal size: launch plane blockIdx.z = b works
// on the matrices at A + b sA, L + b sL, D + b sD, X + b sX with status info[b] (a
// nonzero status on entry skips that matrix in every kernel below).
struct CholBatch {
  int32_t count = 1;
  int64_t sA = 0, sL = 0, sD = 0, sX = 0;
};
// clear_upper: zero each L first (its blocks above the diagonal are never written).
// X: factor [A; I] instead (each plane of A holds 2n rows, sA >= 2 lda n, rows n.. the
// identity, written by the caller), whose identity rows' panels give X = L^-1
// (lower, zero above the diagonal; planes at sX) with no separate triangular inverse
hipError_t chol_factor_batched(double *A, int32_t lda, double *L, int32_t ldl, double *D,
                               int32_t n, int32_t *info, const CholBatch &bt, hipStream_t s,
                               bool clear_upper = true, double *X = nullptr, int32_t ldx = 0);

// out = X^T X (full symmetric) for lower-triangular X on fp64 MFMA: the upper parts of
// X's diagonal blocks must hold zeros, its blocks above the diagonal are never read;
// per batch matrix b at X + b sX and out + b sA (chol.hip)
hipError_t launch_ata_batched(const double *X, int32_t ld, double *out, int32_t n,
                              const int32_t *info, const CholBatch &bt, hipStream_t s);
hipError_t chol_factor(double *A, int32_t lda, double *L, int32_t ldl, double *D, int32_t n,
                       int32_t *info, hipStream_t s, int32_t n_extra = 0, double *LE = nullptr,
                       int32_t ldle = 0, const int32_t *halt = nullptr, bool clear_upper = true,
                       int32_t n_ident = 0, bool first_block_done = false);

hipError_t launch_copy_matrix(const double *src, int32_t lds, double *dst, int32_t ldd, int32_t n,
                              hipStream_t s);
// dst (2n x n, row stride n) = [src; I] (chol.hip)
hipError_t launch_copy_ident(const double *src, int32_t lds, double *dst, int32_t n,
                             hipStream_t s);
// y = A^T x for an upper-triangular n x n A
hipError_t launch_gemv_t_upper(const double *A, int32_t ld, const double *x, double *y, int32_t n,
                               hipStream_t s);
hipError_t launch_tril_copy(const double *src, double *dst, int32_t ld, int32_t n,
                            hipStream_t s);
hipError_t launch_transpose(const double *src, double *dst, int32_t ld, int32_t n,
                            hipStream_t s);
hipError_t launch_gemv_rows(const double *A, int32_t ld, const double *x, double *y,
                            int32_t n, int32_t lower, hipStream_t s);
hipError_t launch_ata_lower(const double *X, int32_t ld, double *out, int32_t n,
                            hipStream_t s);
hipError_t launch_reduce_min(const double *x, int32_t n, double *out, hipStream_t s);
// Newton iteration of the Laplace classifier. Every kernel taking `halt` returns at once
// when *halt != 0 (set at the end of an iteration), so that iterations can be enqueued
// before the previous one's convergence is known.
struct NewtonStatus {
  double delta;  // max |f_new - f| of the iteration
  int32_t info;  // factorisation info after the iteration
  int32_t halt;  // 0 go on, 1 converged, 2 step not finite, 3 factorisation failed
};
// Device counters of the end-of-iteration reduction (zero before the first iteration;
// the last workgroup of every iteration clears them again).
struct NewtonScratch {
  unsigned long long dmax;  // bits of max |f_new - f| (non-negative doubles order as integers)
  unsigned int ticket;      // workgroups done
  unsigned int pad;
};
// Probit likelihood log Phi(t f) (labels t = +-1): grad = t phi(f) / Phi(t f) and
// W = -d2/df2 = r^2 + t f r with r = phi(f) / Phi(t f) = sqrt(2/pi) / erfcx(-t f / sqrt2),
// stable for all t f.
__device__ inline void probit_terms(double f, double t, double &g, double &w) {
  const double z = t * f;
  const double r = 0.79788456080286535588 / erfcx(-z * 0.70710678118654752440);
  g = t * r;
  w = r * r + z * r;
}
// Setup of one Newton iteration at f (chol.hip): probit terms grad, W, sw = W^1/2 and
// b = W f + grad (n each), v = W^1/2 K b, the stacked factorisation input A = [B ; I]
// (2n rows, leading dimension n) with B = I + W^1/2 K W^1/2, and, in one more
// workgroup, the factorisation of B's first diagonal block into L and D[0] (what
// chol_factor's first launch would do; failing pivot into *info).
hipError_t launch_newton_setup(const double *K, const double *f, const double *t, double *grad,
                               double *W, double *sw, double *b, double *v, double *A, int32_t n,
                               double *L, double *D, int32_t *info, const int32_t *halt,
                               hipStream_t s);
// Partial sums y[s][c] = sum_{r in row slice s} A[r][c] x[r] for c < n over kGemvSlices
// equal row slices (y holds kGemvSlices x n; halt may be null).
constexpr int kGemvSlices = 4;
hipError_t launch_gemv_cols(const double *A, int32_t ld, const double *x, double *y, int32_t m,
                            int32_t n, const int32_t *halt, hipStream_t s);
// a = b - sw * (Y z) for the upper triangular Y (n x n, row-major) and z the sum of the
// kGemvSlices partial rows of launch_gemv_cols' output (a may be b; nothing once *halt).
hipError_t launch_newton_a(const double *Y, const double *zs, const double *b, const double *sw,
                           double *a, int32_t n, const int32_t *halt, hipStream_t s);
// End of a Newton iteration: y = K b (n x n K, leading dimension ld), then
// delta = max_r |y[r] - f[r]|; the last workgroup sets *halt (1 once delta < tol, 2 if
// delta is not finite, 3 if *info reports a failed factorisation) and writes the
// iteration's status to *st (host-visible memory).
hipError_t launch_gemv_newton(const double *K, const double *b, double *y, const double *f,
                              int32_t ld, int32_t n, double tol, const int32_t *info,
                              int32_t *halt, NewtonScratch *scr, NewtonStatus *st,
                              hipStream_t s);
// Packed B^T for the contraction in the split fp16 layout: column c < nsrc of B holds
// scale * X[c][k] * rowscale[k] for k <= c (zero elsewhere and for c >= nsrc), where X is
// the lower triangular Linv, or the transpose of the upper triangular Linv when
// `transposed`; each column gets its own power-of-two scale, folded with 2^kexp into
// cscale[c].
hipError_t launch_pack_bt(const double *Linv, int32_t ldl, int32_t nsrc, bool transposed,
                          const double *rowscale, double scale, int32_t kexp, uint16_t *Bt,
                          float *cscale, int32_t ldb, int32_t ncols_pad, hipStream_t s);
// The same layout for one dense column scale * v[k] (k < n), followed by ncols_pad - 1
// zero columns.
hipError_t launch_pack_vec(const double *v, int32_t n, double scale, int32_t kexp, uint16_t *Bt,
                           float *cscale, int32_t ldb, int32_t ncols_pad, hipStream_t s);

hipError_t launch_gather_f64(const double *src, const int32_t *idx, double *dst, int32_t n,
                             hipStream_t s);
hipError_t launch_labels(const uint8_t *feasible, const int32_t *order, double *t, int32_t n,
                         hipStream_t s);

}  // namespace bgp
