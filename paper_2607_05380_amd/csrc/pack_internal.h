// Internal declarations shared by the host runtime and the gfx950 kernels of
// the packed-MLP library: device-side descriptors, launch arguments and the
// kernel launchers.  Nothing here is part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

struct pack_handle;  // the library handle (include/tabpack.h)

namespace tabpack {

constexpr int kChunk = 256;        // AdamW chunk: elements of one member, one kind (weight / bias)
constexpr int kMaxOut = 16;        // largest head width d_out supported by the head kernels
constexpr int kRowAlign = 256;     // base-batch rows are padded to a multiple of this (largest GEMM row tile)
constexpr uint32_t kTagDropout = 3;

// Grouped-GEMM output tiles: big 256 x 256 (4 waves of 128 x 128), tall
// 256 x 128 (4 waves of 128 x 64), small 128 x 128 (4 waves of 64 x 64), and
// for the embedded first layer's forward wide 128 x 256 and tall 256 x 128
// tiles of 8 waves of 64 x 64 (the latter for a last column strip of at most
// 128 columns).
constexpr int kShapeBig = 0, kShapeSmall = 1, kShapeTall = 2, kShapeWide = 3, kShapeTall8 = 4;
constexpr int kBigTile = 256, kSmallTile = 128;
// Tile sets of one launch (one kernel each): big tiles with small edge strips
// (one workgroup per CU), small tiles only, tall tiles with small edge strips
// (two workgroups per CU each), or wide tiles with tall 8-wave tiles for a
// narrow last column strip (one workgroup of 8 waves per CU).
enum TileSet : int { TILES_BIG = 0, TILES_SMALL = 1, TILES_TALL = 2, TILES_WIDE = 3 };
constexpr int kPartRows = 64;   // rows per bias-gradient partial written by the dX epilogue
constexpr int kXcds = 8;        // MI355X: workgroups go round-robin to 8 XCDs
static_assert(kRowAlign % kBigTile == 0, "row padding must cover whole GEMM row tiles");

enum class Prec : int { BF16 = 0, FP32 = 1 };
enum class Task : int { REG = 0, BIN = 1, MULTI = 2 };

// Operand access kinds of the grouped GEMM.  For an operand tile of R rows
// (the GEMM's M or N index) by BK depth (its K index):
//   KMAJ    element (r, k) at P[r * ld + k]         -- depth contiguous
//   RMAJ    element (r, k) at P[k * ld + r]         -- rows contiguous (transposed on load)
//   EMB     the embedded first-layer input E (rows: batch rows, depth: the
//           d_in * d_emb embedding columns), produced inside the GEMM from
//           the member's data rows and embedding parameters (A operand of the
//           first-layer forward of packs with periodic embeddings)
enum OpKind : int { OP_KMAJ = 0, OP_RMAJ = 1, OP_EMB = 2 };
enum EpiKind : int { EPI_FWD = 0, EPI_FWD_EVAL = 1, EPI_DX = 2, EPI_DW = 3, EPI_NS = 4, EPI_DE = 5 };

struct MemberDev;

// One member's GEMM problem C[m, n] = sum_k A(m, k) B(n, k) in one grouped launch.
// most batch rows a weight-gradient GEMM can take straight from the data copy
constexpr int kMapRows = 2048;

struct GemmDesc {
  const void* A;
  const void* B;
  void* C;
  const float* bias;   // EPI_FWD*: [N] fp32
  uint32_t* mask;      // EPI_FWD: written, EPI_DX: read -- ReLU/dropout keep bits of the activation,
                       // word (row/32, col) at mask[(row/32) * N + col], bit row % 32
  const uint32_t* keepw;  // EPI_FWD: dropout keep words of this layer, same layout as mask
  float* colpart;      // EPI_DX: [M / kPartRows, N] column sums of the unrounded output per row block
  int64_t lda, ldb, ldc;
  int32_t M, N, Kd;    // A rows in bounds (< M), B rows in bounds (< N), depth (< Kd)
  int32_t width;       // EPI_FWD*: true width; columns >= width are written as 0
  int32_t member;
  uint32_t drop_t;     // t_k
  float drop_s;        // s_k
  float lr, wd;        // EPI_DW with fused AdamW: the member's learning rate and weight decay
  int32_t pad_;
  int64_t poff;        // EPI_DW with fused AdamW, EPI_NS with the Muon update: element offset of the weight tensor
  const void* Y;       // EPI_NS: the matrix added to the product (GEMM precision), or nullptr
  int64_t ldy;
  // bf16 only: the batch rows of the operand that holds the data, taken
  // straight from a bf16 copy of X (xsrc_rows rows): when xrows is set, batch
  // row r < xrows_n is row xrows[r] of that copy, rows >= xrows_n read as
  // zero.  EPI_FWD: the rows of A (depth-contiguous, lda); EPI_DW: the depth
  // rows of B (rows-contiguous, ldb), at most kMapRows of them.  The embedded
  // first layer's weight gradient (B = OP_EMB, bf16 or fp32) takes its batch
  // rows' data rows from xrows the same way.
  const int32_t* xrows;
  int32_t xrows_n;
  int64_t xsrc_rows;
  // EPI_DW with fused AdamW: the rows r >= opt_rows (past the member's true
  // width) are zero padding, left untouched (their gradients, moments and
  // values stay exactly zero).  The columns' padding is updated like weights:
  // skipping it leaves holes in the rows' streaming stores, which measured
  // slower.
  int32_t opt_rows;
  // EPI_NS with the Muon update: the weight is stored transposed to X (tall);
  // its decay 1 - lr wd and step lr max(1, rows / cols)^(1/2)
  int32_t ns_tall;
  float ns_decay, ns_step;
  int32_t pad3_;
};

struct Tile {
  int32_t desc;
  int32_t m0;
  int32_t n0;
  int32_t shape;       // kShapeBig or kShapeSmall
};

struct AdamConst {
  float beta1, beta2, eps;
  float omb1, omb2;  // 1 - beta1, 1 - beta2, formed in double precision on the host
  float bc1;         // 1 - beta1^t
  float bc2_sqrt;    // sqrt(1 - beta2^t)
};

struct GemmArgs {
  const GemmDesc* descs;
  const Tile* tiles;
  int32_t ntiles;
  int32_t layer;        // 1-based hidden layer (dropout counter)
  int32_t rows_valid;   // batch rows that exist (B in training, chunk rows in eval)
  uint32_t key0, key1;  // dropout stream key
  uint32_t step;        // dropout counter word
  const void* zeros;    // >= 16 bytes of zeros in device memory (source for out-of-range elements)
  int32_t tile_set;     // TileSet of the launch's tiles (selects the kernel)
  // EPI_DW only: when theta is set the epilogue applies AdamW to the weight
  // elements it produces (theta, m, v and the bf16 shadow at desc.poff + the
  // element's index) and stores the gradient itself only if keep_grad is set.
  float* theta;
  float* am;
  float* av;
  uint16_t* shadow;
  AdamConst adam;
  int32_t keep_grad;
  // EPI_NS only: C = ns_alpha * Y + ns_beta * (A B^T), stored in the GEMM precision;
  // with ns_sym the launch holds only tiles on or above the diagonal of a
  // symmetric C and every tile above it also stores its transpose
  float ns_alpha, ns_beta;
  int32_t ns_sym;
  // EPI_NS, the last Newton-Schulz iteration (ns_theta set): instead of
  // storing the new X, the epilogue applies the Muon update to the weight
  // whose X it is, W <- W ns_decay - ns_step O at desc.poff with O = X rounded
  // to the GEMM precision (transposed back for tall weights: desc.ns_tall),
  // and writes the bf16 copy of W to ns_shadow (if set) at the same offsets
  float* ns_theta;
  uint16_t* ns_shadow;
  // EPI_DE only (the embedded first layer's dE = dZ_1 W_1, never stored): the
  // epilogue reduces each wave's 64 rows of dE into the four embedding-gradient
  // terms per column (alpha: dE f, beta: dE, w: -dE alpha sin(phi) x, b:
  // -dE alpha sin(phi); f = x or cos(phi), phi = w x + b) and writes them at
  // C + ((row0 / 64) * 4 + q) * ldc + col.  x of batch row r (< rows_valid) is
  // emb_x[emb_idx[member * rows_valid + r] * emb_d_in + feature]; w, b and
  // alpha come from the column table emb_tab (below).
  const float* emb_x;
  const int32_t* emb_idx;
  const MemberDev* emb_mem;
  int32_t emb_d_in;
  // OP_EMB only (the embedded first layer, E produced in the GEMM from the
  // data and each member's column table emb_tab, see MemberDev::e_tab): x of
  // batch row r is emb_x[row * emb_d_in + feature].  Forward: row =
  // emb_idx[member * rows_valid + r] (training) or emb_row_base + r
  // (emb_idx == nullptr: evaluation and prediction), for r < rows_valid.
  // Weight gradient: row = desc.xrows[r] for r < desc.xrows_n.  emb_x has
  // emb_x_rows rows.
  const float4* emb_tab;
  int64_t emb_row_base;
  int64_t emb_x_rows;
};

// AdamW constants of one step.

// Per-member table used by the small kernels.
struct MemberDev {
  int32_t width, dp;
  uint32_t drop_t;
  float drop_s;
  float lr, wd;
  int64_t act_off;          // member offset inside one activation buffer (elements)
  int64_t w_out_off, b_out_off, b_last_off;  // head weight, head bias, last hidden bias (elements of theta)
  int64_t h_last;           // the member's last hidden activation H_depth: offset from the start of H_1 (elements)
  int64_t dz_last;          // its gradient dZ_depth: offset from the start of the dZ ping-pong pair (elements)
  int32_t depth;            // hidden blocks of the member
  int32_t d_emb;            // periodic embedding size per feature (0: no embedding)
  // periodic embeddings: offsets (elements of theta / grad) of w, b [d_in, d_emb-1]
  // and alpha, beta [d_in, d_emb]; e_act: offset of the member's embedded batch E
  // [Bp, p_in] in the E buffer and of its gradient in the dE buffer
  int64_t e_w, e_b, e_a, e_be, e_act;
  // first entry of the member's embedding column table (float4 units): entry
  // c < p_in holds {w, b, alpha, beta} of column c = i d_emb + j (w = b = 0 for
  // j = 0, zeros for the padding columns); bf16 packs store w and b divided by
  // 2 pi (the phase in revolutions)
  int64_t e_tab;
  int32_t p_in;             // columns of the first layer's input (padded d_in * d_emb, or d_in)
  int32_t pad_;
};

// One hidden weight W [R x Cp] (padded storage, row stride Cp) updated by Muon.
// Its Newton-Schulz iterate X is [S x L] row-major in the GEMM precision:
// X = U (S = R, L = Cp), or X = U^T (S = Cp, L = R) when the weight's true
// rows exceed its true columns (tall).  A and B' are [S x S].
struct MuonMat {
  int64_t woff;    // element offset of W in theta, grad and the momentum buffer
  int64_t xoff;    // element offset of X in each of the two X buffers
  int64_t aoff;    // element offset of A in the A buffer and of B' in the B buffer
  int32_t R, Cp;
  int32_t tall;
  int32_t member;
  float decay;     // 1 - lr wd
  float step;      // lr max(1, rows / cols)^(1/2), true rows and columns
};

struct MuonTile {  // 64 x 64 block (rows r0.., columns c0..) of a MuonMat's W
  int32_t mat, r0, c0, pad_;
};

struct HeadTile {            // (member, first column, first row) block of the head backward
  int32_t member, c0, r0;
};

struct ColTile {            // (member, first column, kind) work item of the gradient sums
  int32_t member;
  int32_t c0;
  int32_t part;             // >= 0: b_{part + 1} from the partials of the dX launch of layer part + 2;
                            // kSumHead: W_out and b_L from the head backward's partials;
                            // kSumLoss: the member's batch-mean loss and b_out (c0 = 0)
};
constexpr int32_t kSumHead = -1, kSumLoss = -2;

// Launchers (kernels_gemm.hip).
hipError_t launch_gemm(Prec prec, OpKind a, OpKind b, EpiKind e, const GemmArgs& args, hipStream_t s);

// Head forward modes: training loss and dY / score-ready eval value / all prediction values.
constexpr int kHeadTrain = 0, kHeadEval = 1, kHeadPredict = 2;

// Launchers (kernels_aux.hip).
hipError_t launch_head_fwd(Prec prec, Task task, int mode, const void* H, const float* theta,
                           const MemberDev* mem, int K, int Bp, int d_out, const void* y,
                           const int32_t* idx, int B, int rows_valid, int64_t row_base, int64_t Nv,
                           float* dY, float* rowloss, float* pred, const int32_t* members, hipStream_t s);
hipError_t launch_head_bwd(Prec prec, const void* H, const float* theta, const MemberDev* mem,
                           const HeadTile* tiles, int ntiles, int Bp, int RB, int d_out, const float* dY,
                           void* dZ, float* part, hipStream_t s);
int head_bwd_cols(int d_out);  // columns one head-backward block covers
// The greedy selection of pack_select() with the caller's scratch `work`
// (pack_select_workspace_size() bytes, 256-byte aligned); returns a PACK_*
// code and sets the library's last error.
int select_with_scratch(pack_handle* h, const float* cand, const void* yv, int32_t C, int64_t Nv, int32_t m_ens,
                        void* work, size_t work_bytes, int32_t* sel_out, int32_t* n_sel_out, double* score_out,
                        hipStream_t stream);
// Sets the library's last error message; returns code.
int set_error(int code, const char* msg);
// The gradient sums of one member group after its last backward launch (one
// wave per ColTile): hidden-layer bias gradients from the dX epilogues'
// partials (bias layer j at colpart + j * part_stride), the head weight and
// last hidden bias gradients from the head backward's partials (RB rows per
// block), and each member's loss (loss_out) and head-bias gradient from the
// per-row losses and dY.  Fixed summation orders.
hipError_t launch_grad_sums(const float* colpart, int64_t part_stride, const float* headpart, int RB,
                            const float* rowloss, const float* dY, const MemberDev* mem, const ColTile* tiles,
                            int ntiles, int Bp, int B, int d_out, const int64_t* bias_off, int K, float* grad,
                            float* loss_out, hipStream_t s);
hipError_t launch_gather(Prec prec, const float* X, int d_in, int Pin, const int32_t* idx, int B,
                         int64_t row_base, int rows_valid, int members, int Bp, void* H0,
                         const int32_t* member_ids, hipStream_t s);
// out[i] = idx[i], or 0 with status[0] = 1 where idx[i] lies outside [0, N)
hipError_t launch_idx_check(const int32_t* idx, int64_t n, int64_t N, int32_t* out, uint32_t* status,
                            hipStream_t s);
// dst <- src, n16 16-byte vectors, non-temporal loads and stores
hipError_t launch_stream_copy(const void* src, void* dst, int64_t n16, hipStream_t s);
// shadow: where the bf16 copy of the updated parameters goes, or nullptr for none
hipError_t launch_adamw(Prec prec, float* theta, const float* grad, float* m, float* v,
                        uint16_t* shadow, const uint32_t* chunk_tab, const uint32_t* list,
                        const MemberDev* mem, int64_t nchunks, const AdamConst& ac, hipStream_t s);
hipError_t launch_to_shadow(const float* theta, uint16_t* shadow, int64_t n, hipStream_t s);
// xb[r][c] = bf16(X[r][c]) for c < d_in, 0 for d_in <= c < Pin; N rows
hipError_t launch_rows_to_bf16(const float* X, int64_t N, int d_in, int Pin, void* xb, hipStream_t s);
// Periodic embeddings (kernels_embed.hip).  The listed members' embedding
// column tables (MemberDev::e_tab) from their
// current parameters in theta; max_pin: the largest first-layer width p_in of
// the listed members (the grid's column extent).
hipError_t launch_embed_table(Prec prec, int d_in, const MemberDev* mem, const int32_t* members, int nmembers,
                              int max_pin, const float* theta, float4* tab, hipStream_t s);
// grad of w, b, alpha, beta from the EPI_DE partial sums (in the dE buffer at
// each member's e_act / 16: [Bp / 64][4][p_in])
hipError_t launch_embed_grad(int d_in, int Bp, const MemberDev* mem, const int32_t* members, int nmembers,
                             int max_pin, const float* part, float* grad, hipStream_t s);
// members: the K member ids whose rows of pred are scored (nullptr: 0 .. K-1)
hipError_t launch_eval_score(Task task, const float* pred, const void* yv, int K, int64_t Nv,
                             double* score_out, const int32_t* members, hipStream_t s);
hipError_t launch_ensemble_mean(const float* part, int n, int Bp, int rows, int d_out, int64_t row_base,
                                float* out, hipStream_t s);
hipError_t launch_dropout_mask(uint32_t key0, uint32_t key1, uint32_t step, int layer, int member,
                               uint32_t t, int B, int width, uint8_t* out, hipStream_t s);
// members: the K member ids to produce words for (nullptr: 0 .. K-1)
hipError_t launch_dropout_words(uint32_t key0, uint32_t key1, uint32_t step, const MemberDev* mem, int K, int L,
                                int max_dp, int Bp, int rows_valid, int64_t A32, uint32_t* out,
                                const int32_t* members, hipStream_t s);
// Muon (kernels_muon.hip): momentum and tile norms, per-matrix inverse norms,
// the normalised (and for tall weights transposed) iterate X0, the update.
hipError_t launch_muon_prep(const MuonMat* mats, const MuonTile* tiles, int ntiles, const float* grad, float* buf,
                            float mu, int nesterov, double* part, hipStream_t s);
hipError_t launch_muon_norm(const int32_t* tile0, int nmats, const double* part, float* inv, hipStream_t s);
hipError_t launch_muon_convert(Prec prec, const MuonMat* mats, const MuonTile* tiles, int ntiles, const float* grad,
                               const float* buf, float mu, int nesterov, const float* inv, void* X, hipStream_t s);
hipError_t launch_muon_update(Prec prec, const MuonMat* mats, const MuonTile* tiles, int ntiles, float* theta,
                              uint16_t* shadow, const void* X, hipStream_t s);
hipError_t launch_select_iter(Task task, const float* cand, const void* yv, int C, int64_t Nv,
                              int m_ens, double* sum, double* partial, int nblk, int32_t* state,
                              double* best, int32_t* sel_out, hipStream_t s);
hipError_t launch_select_init(double* sum, int64_t Nv, int32_t* state, double* best,
                              int32_t* n_sel_out, double* score_out, hipStream_t s);
hipError_t launch_select_final(const int32_t* state, const double* best, int32_t* n_sel_out,
                               double* score_out, hipStream_t s);
int select_blocks(int64_t Nv);

}  // namespace tabpack
