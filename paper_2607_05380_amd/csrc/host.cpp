// Host runtime of the packed-MLP library: argument checking, hyperparameter
// sampling, the packed layout planner, initial parameters, workspace binding,
// launch sequencing of the training step / evaluation / greedy selection, and
// the C ABI declared in include/tabpack.h.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/tabpack.h"
#include "pack_internal.h"
#include "philox.h"

using namespace tabpack;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(PACK_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr uint32_t kTagHparam = 1, kTagInit = 2;
constexpr int kGroups = 4;  // at most this many member groups run their GEMM chains concurrently

int64_t round_up(int64_t x, int64_t q) { return (x + q - 1) / q * q; }

struct Key {
  uint32_t k0, k1;
};
Key stream_key(uint64_t seed, uint32_t tag) {
  return Key{(uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32) ^ (tag << 28)};
}

// Double in [0, 1) with 53 random bits from two 32-bit words.
double u53(uint32_t a, uint32_t b) {
  return ((double)(a >> 5) * 67108864.0 + (double)(b >> 6)) * (1.0 / 9007199254740992.0);
}

double log_uniform(double lo, double hi, double u) {
  if (lo == hi) return lo;
  return std::exp(std::log(lo) + u * (std::log(hi) - std::log(lo)));
}

struct Member {
  int width, dp;
  int depth;  // hidden Linear-ReLU-Dropout blocks, 1 .. L
  double dropout, lr, wd, scale;
  double muon_lr = 0.0;  // Muon learning rate of the hidden weights (Muon packs)
  int d_emb = 0;         // periodic embedding size per feature (0: the features feed W_1 directly)
  double sigma = 0.0;    // standard deviation of the embedding frequencies' initial values
  int p_in = 0;          // columns of W_1 and of the first layer's input (padded d_in * d_emb, or Pin)
  int64_t eoff[4] = {};  // embedding parameters w, b, alpha, beta (offsets in theta)
  int64_t h0_off = 0;    // the member's first-layer input block (elements of the H_0 / E buffer)
  int64_t etab_off = 0;  // the member's embedding column table (entries of the table buffer)
  uint32_t t;
  std::vector<int64_t> toff;  // packed offsets of W_1, b_1, ..., W_depth, b_depth, W_out, b_out
  int64_t act_off;
};

struct Launch {
  int desc0, ndesc;
  int tile0, ntiles;
  double flops;  // algorithmic flops of the launch (true member shapes)
  double bytes;  // algorithmic HBM bytes: operands read once, outputs written once
  TileSet ts = TILES_SMALL;  // tile set of its tiles (set by add_tiles / add_tiles_sym)
};

// One timed launch: events recorded on the launch stream around it.
struct TimedLaunch {
  int group;
  hipEvent_t start, stop;
};

struct ProfGroup {
  std::string name;
  int kind;
  int launches = 0;
  double total_ms = 0.0, flops = 0.0, bytes = 0.0;
};

}  // namespace

// Device buffers carved out of the caller's workspace.
struct Bufs {
  float *theta = nullptr, *grad = nullptr, *m = nullptr, *v = nullptr;
  uint16_t* shadow = nullptr;
  char* H0 = nullptr;  // first-layer inputs: gathered batches [Bp, Pin], or embedded batches E [Bp, p_in], per member
  float4* etab = nullptr;  // embeddings: the members' column tables (MemberDev::e_tab), rebuilt every step
  float* dE = nullptr; // embeddings: at each member's E offset / 16, the dE GEMM's sums [Bp / 64][4][p_in] (fp32)
  char* H = nullptr;   // L activation buffers H_1..H_L
  char* dz = nullptr;  // 2 ping-pong buffers for dZ_l
  float* colpart = nullptr;  // bias-gradient partials of the dX epilogues, (L - 1) x A / kPartRows floats
  uint32_t* mask = nullptr;  // ReLU/dropout keep bits of H_1..H_L, L * A / 32 words
  uint32_t* keepw = nullptr; // dropout keep words, 2 copies of L * A / 32 words
  char* zeros = nullptr;     // 256 zero bytes: GEMM loads of out-of-range elements read them
  float *dY = nullptr, *rowloss = nullptr;
  MemberDev* d_mem = nullptr;
  uint32_t* d_chunks = nullptr;
  uint32_t* d_aux = nullptr;
  int64_t* d_bias_off = nullptr;  // [L][K] offsets of b_l
  GemmDesc* d_descs = nullptr;
  Tile* d_tiles = nullptr;
  size_t tile_cap = 0;  // entries of d_tiles
  ColTile* d_coltiles = nullptr;
  HeadTile* d_headtiles = nullptr;
  int32_t* d_members = nullptr;
  int32_t* d_active = nullptr;  // active member ids, increasing
  // Muon scratch: two X buffers, A, B' (GEMM precision), tile partial norms,
  // inverse norms and the matrix / tile tables
  char* mX[2] = {nullptr, nullptr};
  char* mA = nullptr;
  char* mB = nullptr;
  double* mpart = nullptr;
  float* minv = nullptr;
  MuonMat* d_mmats = nullptr;
  MuonTile* d_mtiles = nullptr;
  int32_t* d_mtile0 = nullptr;
  float* headpart = nullptr;  // head backward partials, (Bp / RB) * (d_out + 1) * A / Bp floats
  int32_t* idx_ok = nullptr;  // the step's batch indices, entries outside [0, N) replaced by 0 [K * B]
  uint32_t* status = nullptr; // asynchronous error flags (pack_status)
};

struct pack_handle {
  pack_config cfg;
  Prec prec;
  Task task;
  int q, Bp, Pin;
  // pack_bind_data: the first layer's forward and weight-gradient GEMMs read
  // the batch rows straight from a bf16 copy of X (xb, data_N rows of Pin)
  // through the batch indices; no H_0 is gathered
  bool stream_rows = false;
  const float* data_X = nullptr;
  int64_t data_N = 0;
  void* xb = nullptr;
  std::vector<Member> mem;
  int64_t P = 0;     // packed parameter count (multiple of kChunk)
  int64_t A = 0;     // elements of one activation buffer (all members)
  std::vector<float> theta_host;  // host copy of the parameters, packed layout
  std::vector<uint32_t> chunk_tab;
  std::vector<uint32_t> aux_chunks;  // chunks the separate AdamW pass updates (biases, head)
  // Members in the pack's launches (Section 3.6: a base model that stops
  // improving is removed from the pack); inactive members keep their state.
  std::vector<uint8_t> active;
  std::vector<int32_t> active_ids;   // increasing
  int64_t n_aux_active = 0;          // aux chunks of active members (uploaded first in d_aux)
  bool muon = false;                 // hidden weights on Muon (pack_config.optimizer)
  bool emb = false;                  // periodic feature embeddings (pack_config.emb_lo > 0)
  Launch de[kGroups]{};
  int ns_steps = 5;
  int n_mmats = 0, n_mtiles = 0;     // Muon matrices and tiles of the active members
  // per member group g: matrices [mmat0[g], mmat0[g+1]), tiles [mtileg[g], mtileg[g+1])
  int mmat0[kGroups + 1]{}, mtileg[kGroups + 1]{};
  Launch nsA[2][kGroups]{}, nsB[kGroups]{}, nsX[2][kGroups]{};

  bool bound = false;
  Bufs b;
  // per layer (index l-1); the forward launches exist once per keep-word
  // buffer: the dropout keep words alternate between two copies by step
  // parity, so the next step's are produced while this step's backward runs
  std::vector<Launch> fwd[2][kGroups], dx[kGroups], dw[kGroups];  // [keep-word parity][group] / [group]
  Launch fwd1_eval{};                // layer 1 over the shared validation rows in H_0 block 0
  // The members are split into ngroups groups of about equal GEMM work; each
  // group's GEMM chain runs on its own stream (group 0 on the caller's), which
  // measured faster than one launch over all members.
  int ngroups = 1;
  std::vector<int> group[kGroups];
  int sumtile0[kGroups + 1] = {};    // gradient-sum work items of group g: [sumtile0[g], sumtile0[g + 1])
  int headtile0[kGroups + 1] = {};   // head-backward tiles of group g
  int member0[kGroups + 1] = {};     // group g's members: d_members[member0[g] .. member0[g+1])
  hipStream_t gstream[kGroups] = {};  // streams of groups 1.. (entry 0 unused)
  hipEvent_t ev_split = nullptr, ev_merge[kGroups] = {};
  hipEvent_t ev_gather[kGroups] = {};  // group g's gather done (group g + 1 gathers after it)
  hipEvent_t ev_bias[kGroups] = {};    // group g's last backward producer done (its gradient sums follow)
  int ncoltiles = 0;
  int nheadtiles = 0;
  int head_rb = 0;  // rows per head-backward block
  uint64_t t = 0;
  TileSet tiles = TILES_SMALL;  // tile set of the bf16 GEMMs (fp32 GEMMs run small tiles only)
  // tile sets of the forward, data- and weight-gradient GEMMs: -1 chooses per
  // launch (launch_tiles), else a fixed TileSet
  int tiles_fwd = -1, tiles_dx = -1, tiles_dw = -1;
  TileSet ns_tiles = TILES_SMALL;  // tile set of the Newton-Schulz GEMMs
  TileSet emb_tiles = TILES_SMALL;  // tile set of the embedded first layer's forward (training and evaluation)
  bool muon_fused = true;  // the Muon update in the last Newton-Schulz GEMM's epilogue
  // side stream for ALU-bound work that overlaps memory-bound kernels of the
  // caller's stream, joined back through events (created by pack_bind)
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  hipEvent_t ev_keep[2] = {nullptr, nullptr};  // keep words of the step with that parity are ready
  uint64_t keep_ready = 0;                     // step whose keep words are (being) produced ahead

  // optional per-kernel timing
  bool prof = false;
  std::vector<TimedLaunch> timed;
  std::vector<hipEvent_t> event_pool;
  size_t pool_used = 0;
  std::vector<ProfGroup> groups;

  size_t elt() const { return prec == Prec::BF16 ? 2 : 4; }
  void* Hl(int l) const { return b.H + (size_t)(l - 1) * A * elt(); }  // H_l, l = 1..L
  int64_t H0e = 0;  // elements of the H_0 / E buffer (every member's first-layer input block)
  int64_t Etab = 0; // entries of the embedding column tables (p_in per embedded member)
  void* dzb(int l) const { return b.dz + (size_t)(l & 1) * A * elt(); } // buffer holding dZ_l
};

namespace {

int validate(const pack_config* c) {
  if (!c) return fail(PACK_EINVAL, "cfg is NULL");
  if (c->K < 1 || c->K > 65535) return fail(PACK_EINVAL, "K=%d out of [1, 65535]", c->K);
  if (c->d_in < 1 || c->d_in > (1 << 20)) return fail(PACK_EINVAL, "d_in=%d out of range", c->d_in);
  if (c->L < 1 || c->L > 8) return fail(PACK_EINVAL, "L=%d out of [1, 8]", c->L);
  if (!(c->depth_lo == 0 && c->depth_hi == 0) && !(1 <= c->depth_lo && c->depth_lo <= c->depth_hi && c->depth_hi <= c->L))
    return fail(PACK_EINVAL, "depth range [%d, %d] must lie in [1, L=%d] (0, 0: every member has L blocks)",
                c->depth_lo, c->depth_hi, c->L);
  if (c->B < 1 || c->B > 65536) return fail(PACK_EINVAL, "B=%d out of [1, 65536]", c->B);
  if (c->task < 0 || c->task > 2) return fail(PACK_EINVAL, "unknown task %d", c->task);
  if (c->precision != PACK_PREC_BF16 && c->precision != PACK_PREC_FP32)
    return fail(PACK_EINVAL, "unknown precision %d", c->precision);
  if (c->task == PACK_TASK_MULTI_CE) {
    if (c->d_out < 2 || c->d_out > kMaxOut) return fail(PACK_EINVAL, "CE needs 2 <= d_out <= %d", kMaxOut);
  } else if (c->d_out != 1) {
    return fail(PACK_EINVAL, "MSE/BCE tasks need d_out == 1");
  }
  const int q = c->quantum ? c->quantum : 32;
  if (q < 8 || q > 512 || q % 8) return fail(PACK_EINVAL, "quantum %d must be a multiple of 8 in [8, 512]", q);
  if (c->keep_grads != 0 && c->keep_grads != 1) return fail(PACK_EINVAL, "keep_grads must be 0 or 1");
  if (!(c->beta1 >= 0 && c->beta1 < 1 && c->beta2 >= 0 && c->beta2 < 1 && c->eps > 0))
    return fail(PACK_EINVAL, "AdamW constants out of range");
  if (c->emb_lo != 0) {
    if (c->emb_lo < 8 || c->emb_hi < c->emb_lo || c->emb_hi > 32 || c->emb_step < 1 ||
        (c->emb_hi - c->emb_lo) % c->emb_step)
      return fail(PACK_EINVAL, "embedding size range [%d, %d] step %d invalid (8 <= lo <= hi <= 32)", c->emb_lo,
                  c->emb_hi, c->emb_step);
    if (!c->members && !(c->sigma_lo > 0 && c->sigma_hi >= c->sigma_lo))
      return fail(PACK_EINVAL, "embedding sigma range must be positive and ordered");
    if (c->B > kMapRows)
      return fail(PACK_EINVAL, "B=%d: periodic embeddings take batches of at most %d rows", c->B, kMapRows);
  }
  if (c->optimizer != PACK_OPT_ADAMW && c->optimizer != PACK_OPT_MUON)
    return fail(PACK_EINVAL, "unknown optimizer %d", c->optimizer);
  if (c->optimizer == PACK_OPT_MUON) {
    if (c->ns_steps < 0 || c->ns_steps > 16) return fail(PACK_EINVAL, "ns_steps=%d out of [1, 16]", c->ns_steps);
    if (!(c->muon_momentum >= 0 && c->muon_momentum < 1)) return fail(PACK_EINVAL, "Muon momentum out of [0, 1)");
    if (!c->members && !(c->muon_lr_lo > 0 && c->muon_lr_hi >= c->muon_lr_lo))
      return fail(PACK_EINVAL, "Muon learning-rate range must be positive and ordered");
  }
  if (!c->members) {
    if (c->width_lo < 1 || c->width_hi < c->width_lo || c->width_hi > 16384)
      return fail(PACK_EINVAL, "width range [%d, %d] invalid", c->width_lo, c->width_hi);
    if (!(c->dropout_lo >= 0 && c->dropout_hi >= c->dropout_lo && c->dropout_hi < 1))
      return fail(PACK_EINVAL, "dropout range invalid");
    if (!(c->lr_lo > 0 && c->lr_hi >= c->lr_lo) || !(c->wd_lo > 0 && c->wd_hi >= c->wd_lo))
      return fail(PACK_EINVAL, "lr/wd ranges must be positive and ordered");
  }
  return PACK_OK;
}

void sample_members(pack_handle* h) {
  const pack_config& c = h->cfg;
  const Key key = stream_key(c.seed, kTagHparam);
  for (int k = 0; k < c.K; ++k) {
    const Words4 a = philox4x32_10((uint32_t)k, 0, 0, 0, key.k0, key.k1);
    const Words4 b = philox4x32_10((uint32_t)k, 1, 0, 0, key.k0, key.k1);
    Member& m = h->mem[k];
    m.width = c.width_lo + (int)std::floor(u53(a.w0, a.w1) * (double)(c.width_hi - c.width_lo + 1));
    m.dropout = c.dropout_lo + u53(a.w2, a.w3) * (c.dropout_hi - c.dropout_lo);
    m.lr = log_uniform(c.lr_lo, c.lr_hi, u53(b.w0, b.w1));
    m.wd = log_uniform(c.wd_lo, c.wd_hi, u53(b.w2, b.w3));
    m.depth = c.L;
    if (c.depth_lo > 0) {  // depth ~ UniformInt[depth_lo, depth_hi] from block (k, 2, 0, 0)
      const Words4 d = philox4x32_10((uint32_t)k, 2, 0, 0, key.k0, key.k1);
      m.depth = c.depth_lo + (int)std::floor(u53(d.w0, d.w1) * (double)(c.depth_hi - c.depth_lo + 1));
    }
    if (c.optimizer == PACK_OPT_MUON) {  // Muon learning rate from block (k, 3, 0, 0)
      const Words4 d = philox4x32_10((uint32_t)k, 3, 0, 0, key.k0, key.k1);
      m.muon_lr = log_uniform(c.muon_lr_lo, c.muon_lr_hi, u53(d.w0, d.w1));
    }
    if (c.emb_lo > 0) {  // embedding size and sigma from block (k, 4, 0, 0)
      const Words4 d = philox4x32_10((uint32_t)k, 4, 0, 0, key.k0, key.k1);
      m.d_emb = c.emb_lo + c.emb_step * (int)std::floor(u53(d.w0, d.w1) * (double)((c.emb_hi - c.emb_lo) / c.emb_step + 1));
      m.sigma = log_uniform(c.sigma_lo, c.sigma_hi, u53(d.w2, d.w3));
    }
  }
}

// Packed layout: per member, tensors W_1 [dp, Pin], b_1 [dp], W_l [dp, dp],
// b_l [dp], W_out [d_out, dp], b_out [d_out]; every tensor starts on a
// kChunk-element boundary so an AdamW chunk never mixes members or
// weights with biases.  Padding rows/columns hold exact zeros forever: their
// inputs or output gradients are zero, so their gradients and AdamW moments
// stay zero.
int emb_dp(int d_emb) { return (d_emb + 7) & ~7; }

void plan_layout(pack_handle* h) {
  const pack_config& c = h->cfg;
  int64_t off = 0, aoff = 0;
  h->chunk_tab.clear();
  h->aux_chunks.clear();
  int64_t h0 = 0, tab = 0;
  for (int k = 0; k < c.K; ++k) {
    Member& m = h->mem[k];
    m.dp = (int)round_up(m.width, h->q);
    // embedded: feature i owns columns i dp .. i dp + dp - 1 of W_1 (dp = d_emb
    // rounded up to 8, the last dp - d_emb zero padding), so that every
    // 16-byte chunk of a row the GEMMs produce belongs to one feature
    m.p_in = m.d_emb ? c.d_in * emb_dp(m.d_emb) : h->Pin;
    m.h0_off = h0;
    h0 += (int64_t)h->Bp * m.p_in;
    m.etab_off = tab;
    if (m.d_emb) tab += m.p_in;
    if (m.d_emb) {  // embedding parameters first: w, b [d_in, d_emb-1], alpha, beta [d_in, d_emb] (AdamW)
      const int64_t n[4] = {(int64_t)c.d_in * (m.d_emb - 1), (int64_t)c.d_in * (m.d_emb - 1),
                            (int64_t)c.d_in * m.d_emb, (int64_t)c.d_in * m.d_emb};
      for (int t = 0; t < 4; ++t) {
        m.eoff[t] = off;
        const int64_t nc = round_up(n[t], kChunk) / kChunk;
        for (int64_t i = 0; i < nc; ++i) {
          h->aux_chunks.push_back((uint32_t)h->chunk_tab.size());
          h->chunk_tab.push_back((uint32_t)k);
        }
        off += nc * kChunk;
      }
    }
    m.toff.assign(2 * m.depth + 2, 0);
    for (int l = 0; l <= m.depth; ++l) {
      const int64_t rows = l < m.depth ? m.dp : c.d_out;
      const int64_t cols = l == 0 ? m.p_in : m.dp;
      for (int part = 0; part < 2; ++part) {
        const int64_t n = part == 0 ? rows * cols : rows;
        m.toff[2 * l + part] = off;
        const int64_t nc = round_up(n, kChunk) / kChunk;
        const uint32_t flag = (part == 1 && !c.decay_bias) ? 0x80000000u : 0u;
        // hidden-layer weights are updated inside their weight-gradient GEMM
        const bool fused = part == 0 && l < m.depth;
        for (int64_t i = 0; i < nc; ++i) {
          if (!fused) h->aux_chunks.push_back((uint32_t)h->chunk_tab.size());
          h->chunk_tab.push_back((uint32_t)k | flag);
        }
        off += nc * kChunk;
      }
    }
    m.act_off = aoff;
    aoff += (int64_t)h->Bp * m.dp;
  }
  h->P = off;
  h->A = aoff;
  h->H0e = h0;
  h->Etab = tab;
}

// Packed column of dense column cc (feature-major i d_emb + j) of W_1.
int64_t w1_col(const Member& m, int64_t cc) {
  return m.d_emb ? (cc / m.d_emb) * emb_dp(m.d_emb) + cc % m.d_emb : cc;
}

// torch.nn.Linear default initialisation, U(-1/sqrt(fan_in), 1/sqrt(fan_in)),
// drawn from the init stream: element e of tensor t of member k uses word
// (e & 3) of block (e >> 2, e >> 34, t, k); u = (word >> 8) * 2^-24.
void init_params(pack_handle* h) {
  const pack_config& c = h->cfg;
  h->theta_host.assign((size_t)h->P, 0.0f);
  const Key key = stream_key(c.seed, kTagInit);
  for (int k = 0; k < c.K; ++k) {
    const Member& m = h->mem[k];
    if (m.d_emb) {
      // embedding frequencies w ~ N(0, sigma) by Box-Muller: element e takes block
      // (e >> 1, 0, 100, k); u1 = ((word0 >> 8) + 1) 2^-24, u2 = (word1 >> 8) 2^-24;
      // cos for even e, sin for odd e.  b, alpha, beta start at zero.
      const int64_t n = (int64_t)c.d_in * (m.d_emb - 1);
      float* dst = h->theta_host.data() + m.eoff[0];
      for (int64_t e = 0; e < n; ++e) {
        const Words4 w = philox4x32_10((uint32_t)(e >> 1), 0, 100, (uint32_t)k, key.k0, key.k1);
        const double u1 = (double)((w.w0 >> 8) + 1) * (1.0 / 16777216.0);
        const double u2 = (double)(w.w1 >> 8) * (1.0 / 16777216.0);
        const double r = std::sqrt(-2.0 * std::log(u1));
        const double z = r * ((e & 1) == 0 ? std::cos(2.0 * M_PI * u2) : std::sin(2.0 * M_PI * u2));
        dst[e] = (float)(m.sigma * z);
      }
    }
    for (int l = 0; l <= m.depth; ++l) {
      const int rows = l < m.depth ? m.width : c.d_out;
      const int fan_in = l == 0 ? (m.d_emb ? c.d_in * m.d_emb : c.d_in) : m.width;
      const int64_t ld = l == 0 ? m.p_in : m.dp;
      const double bound = 1.0 / std::sqrt((double)fan_in);
      for (int part = 0; part < 2; ++part) {
        const uint32_t tid = (uint32_t)(2 * l + part);
        const int64_t n = part == 0 ? (int64_t)rows * fan_in : rows;
        float* dst = h->theta_host.data() + m.toff[2 * l + part];
        Words4 w{};
        for (int64_t e = 0; e < n; ++e) {
          if ((e & 3) == 0 || e == 0)
            w = philox4x32_10((uint32_t)(e >> 2), (uint32_t)(e >> 34), tid, (uint32_t)k, key.k0, key.k1);
          const uint32_t word = (e & 3) == 0 ? w.w0 : (e & 3) == 1 ? w.w1 : (e & 3) == 2 ? w.w2 : w.w3;
          const double u = (double)(word >> 8) * (1.0 / 16777216.0);
          const float val = (float)((2.0 * u - 1.0) * bound);
          if (part == 0)
            dst[(e / fan_in) * ld + (l == 0 ? w1_col(m, e % fan_in) : e % fan_in)] = val;
          else
            dst[e] = val;
        }
      }
    }
  }
}

// Dense <-> packed copies of one member's tensors.
int64_t dense_count(const pack_handle* h, int k) {
  const Member& m = h->mem[k];
  const pack_config& c = h->cfg;
  const int64_t fi = m.d_emb ? (int64_t)c.d_in * m.d_emb : c.d_in;
  const int64_t emb = m.d_emb ? 2 * (int64_t)c.d_in * (2 * m.d_emb - 1) : 0;
  return emb + (int64_t)m.width * fi + m.width + (int64_t)(m.depth - 1) * ((int64_t)m.width * m.width + m.width) +
         (int64_t)c.d_out * m.width + c.d_out;
}

template <typename F>
void for_each_dense(const pack_handle* h, int k, F f) {  // f(dense_index, packed_index)
  const Member& m = h->mem[k];
  const pack_config& c = h->cfg;
  int64_t di = 0;
  if (m.d_emb) {  // embedding parameters first: w, b [d_in, d_emb-1], alpha, beta [d_in, d_emb]
    const int64_t n[4] = {(int64_t)c.d_in * (m.d_emb - 1), (int64_t)c.d_in * (m.d_emb - 1),
                          (int64_t)c.d_in * m.d_emb, (int64_t)c.d_in * m.d_emb};
    for (int t = 0; t < 4; ++t)
      for (int64_t e = 0; e < n[t]; ++e) f(di++, m.eoff[t] + e);
  }
  for (int l = 0; l <= m.depth; ++l) {
    const int rows = l < m.depth ? m.width : c.d_out;
    const int cols = l == 0 ? (m.d_emb ? c.d_in * m.d_emb : c.d_in) : m.width;
    const int64_t ld = l == 0 ? m.p_in : m.dp;
    for (int r = 0; r < rows; ++r)
      for (int cc = 0; cc < cols; ++cc) f(di++, m.toff[2 * l] + (int64_t)r * ld + (l == 0 ? w1_col(m, cc) : cc));
    for (int r = 0; r < rows; ++r) f(di++, m.toff[2 * l + 1] + r);
  }
}

int64_t member_span_begin(const pack_handle* h, int k) {
  return h->mem[k].d_emb ? h->mem[k].eoff[0] : h->mem[k].toff[0];
}
int64_t member_span_end(const pack_handle* h, int k) {
  return k + 1 < h->cfg.K ? member_span_begin(h, k + 1) : h->P;
}

// Device-table sizes.
struct Plan {
  TileSet tile_set = TILES_SMALL;
  std::vector<GemmDesc> descs;
  std::vector<Tile> tiles;
  std::vector<int64_t> cost;  // planner's cost of each tile (depth x valid area)
  std::vector<ColTile> coltiles;
  std::vector<HeadTile> headtiles;
  std::vector<Launch> fwd[2][kGroups], dx[kGroups], dw[kGroups];
  Launch fwd1_eval{};
  int sumtile0[kGroups + 1] = {};  // see build_plan
  int headtile0[kGroups + 1] = {};
  std::vector<int32_t> members;  // member ids in group order
  int member0[kGroups + 1] = {};
  // Muon: the hidden weights, their 64 x 64 tiles (matrix k owns tiles
  // mtile0[k] .. mtile0[k+1]) and the Newton-Schulz products: A = X X^T and
  // X' = a X + B' X for each parity of the X buffers, B' = b A + c A A
  std::vector<MuonMat> mmats;
  std::vector<MuonTile> mtiles;
  std::vector<int32_t> mtile0;
  int mmat0[kGroups + 1]{}, mtileg[kGroups + 1]{};  // per member group: first matrix, first tile
  Launch nsA[2][kGroups]{}, nsB[kGroups]{}, nsX[2][kGroups]{};
  // embeddings: dE = dZ_1 W_1 per group (the first layer's data gradient,
  // reduced in the epilogue into the embedding-gradient sums)
  Launch de[kGroups]{};
};

// Tiles of one member's M x N output.  Big set: 256 x 256 tiles, except that
// a remainder of at most 128 rows or columns is covered by a strip of small
// 128 x 128 tiles (a larger remainder takes one more, partly filled, big
// tile).  Tall set: 256 x 128 tiles, rows as in the big set, the last column
// tile partly filled.  Small set: 128 x 128 tiles only.
void add_tiles(Plan& p, Launch& ln, int d, int M, int N, int kdepth) {
  const size_t first = p.tiles.size();
  ln.ts = p.tile_set;
  auto big_end = [&](int E) {
    const int r = E % kBigTile;
    return r == 0 ? E : (r > kSmallTile ? E - r + kBigTile : E - r);
  };
  if (p.tile_set == TILES_WIDE) {
    // 128 x 256 tiles; a last strip of at most 128 columns on 256 x 128 tiles
    const int r = N % kBigTile, Nw = r > 0 && r <= kSmallTile ? N - r : N;
    for (int m0 = 0; m0 < M; m0 += kSmallTile)
      for (int n0 = 0; n0 < Nw; n0 += kBigTile) {
        p.tiles.push_back(Tile{d, m0, n0, kShapeWide});
        p.cost.push_back((int64_t)kdepth * std::min(kSmallTile, M - m0) * std::min(kBigTile, N - n0));
      }
    if (Nw < N)
      for (int m0 = 0; m0 < M; m0 += kBigTile) {
        p.tiles.push_back(Tile{d, m0, Nw, kShapeTall8});
        p.cost.push_back((int64_t)kdepth * std::min(kBigTile, M - m0) * (N - Nw));
      }
    ln.ntiles = (int)p.tiles.size() - ln.tile0;
    return;
  }
  const bool big = p.tile_set == TILES_BIG, tall = p.tile_set == TILES_TALL;
  const int Mb = big || tall ? big_end(M) : 0;
  const int Nb = big ? big_end(N) : (tall ? (int)round_up(N, kSmallTile) : 0);
  const int tn = big ? kBigTile : kSmallTile;  // columns of the large tile
  const int large = big ? kShapeBig : kShapeTall;
  auto push = [&](int m0, int n0, int shape) {
    const int tm = shape == kShapeSmall ? kSmallTile : kBigTile;
    const int tw = shape == kShapeBig ? kBigTile : kSmallTile;
    const int mb = std::min(tm, M - m0), nb = std::min(tw, N - n0);
    p.tiles.push_back(Tile{d, m0, n0, shape});
    p.cost.push_back((int64_t)kdepth * std::max(mb, 0) * std::max(nb, 0));
  };
  for (int m0 = 0; m0 < Mb; m0 += kBigTile)
    for (int n0 = 0; n0 < Nb; n0 += tn) push(m0, n0, large);
  for (int m0 = 0; m0 < Mb; m0 += kSmallTile)
    for (int n0 = Nb; n0 < N; n0 += kSmallTile) push(m0, n0, kShapeSmall);
  for (int m0 = Mb; m0 < M; m0 += kSmallTile)
    for (int n0 = 0; n0 < N; n0 += kSmallTile) push(m0, n0, kShapeSmall);
  // Wider than tall (the embedded first layer's dE = dZ_1 W_1 and dW_1 =
  // dZ_1^T E, thousands of columns): tiles in column-strip order, so the row
  // tiles sharing a strip of the wide operand run together and read it once
  // while the narrow operand stays in L2 (row order re-reads every strip once
  // per row tile).
  if (N > M) {
    std::vector<std::pair<Tile, int64_t>> v;
    for (size_t i = first; i < p.tiles.size(); ++i) v.push_back({p.tiles[i], p.cost[i]});
    std::stable_sort(v.begin(), v.end(), [](const std::pair<Tile, int64_t>& x, const std::pair<Tile, int64_t>& y) {
      return x.first.n0 != y.first.n0 ? x.first.n0 < y.first.n0 : x.first.m0 < y.first.m0;
    });
    for (size_t i = 0; i < v.size(); ++i) {
      p.tiles[first + i] = v[i].first;
      p.cost[first + i] = v[i].second;
    }
  }
  ln.ntiles = (int)p.tiles.size() - ln.tile0;
}

// Launch order of one grouped GEMM.  Workgroup i runs on XCD i % 8, and each
// XCD has its own L2, so all tiles of a member go to one XCD (members are
// packed into the 8 XCD bins longest-first by total cost), and within a bin
// tiles run longest-first so the launch ends on short tiles.
void sort_launch(Plan& p, const Launch& ln) {
  struct Item {
    Tile t;
    int64_t cost;
  };
  std::vector<Item> items;
  for (int i = 0; i < ln.ntiles; ++i) items.push_back(Item{p.tiles[ln.tile0 + i], p.cost[ln.tile0 + i]});
  std::vector<std::pair<int64_t, int>> member_cost;  // (cost, desc)
  for (const Item& it : items) {
    auto f = std::find_if(member_cost.begin(), member_cost.end(),
                          [&](const std::pair<int64_t, int>& e) { return e.second == it.t.desc; });
    if (f == member_cost.end())
      member_cost.push_back({it.cost, it.t.desc});
    else
      f->first += it.cost;
  }
  std::stable_sort(member_cost.begin(), member_cost.end(),
                   [](const std::pair<int64_t, int>& a, const std::pair<int64_t, int>& b) { return a.first > b.first; });
  std::vector<int64_t> load(kXcds, 0);
  std::vector<int> bin_of(p.descs.size() + 1, 0);
  for (const auto& mc : member_cost) {
    const int b = (int)(std::min_element(load.begin(), load.end()) - load.begin());
    load[b] += mc.first;
    bin_of[mc.second] = b;
  }
  std::vector<std::vector<Item>> bins(kXcds);
  for (const Item& it : items) bins[bin_of[it.t.desc]].push_back(it);
  for (auto& b : bins)
    std::stable_sort(b.begin(), b.end(), [](const Item& x, const Item& y) { return x.cost > y.cost; });
  std::vector<size_t> next(kXcds, 0);
  for (int i = 0; i < ln.ntiles; ++i) {
    int b = i % kXcds;
    if (next[b] == bins[b].size()) {  // this XCD's bin is empty: take from the fullest remaining
      size_t best = 0;
      for (int c = 0; c < kXcds; ++c)
        if (bins[c].size() - next[c] > best) best = bins[c].size() - next[c], b = c;
    }
    p.tiles[ln.tile0 + i] = bins[b][next[b]].t;
    p.cost[ln.tile0 + i] = bins[b][next[b]].cost;
    ++next[b];
  }
}

// Members into ngroups groups of about equal GEMM work (longest first, each
// to the lightest group).  Default: 2 groups, 3 with Muon, whose per-group
// Newton-Schulz chains overlap better in three (regression_large: 1.398
// against 1.409 ms per step, Muon 5.33 against 5.39 ms; one group 1.53 ms;
// 4 groups exceed the four hardware queues).  TABPACK_STREAMS (1 .. 4)
// overrides it.
void split_members(pack_handle* h) {
  int ng = h->muon ? 3 : 2;
  if (const char* e = getenv("TABPACK_STREAMS")) ng = std::max(1, std::min(kGroups, atoi(e)));
  h->ngroups = std::max(1, std::min(ng, (int)h->active_ids.size()));
  for (auto& v : h->group) v.clear();
  std::vector<std::pair<double, int>> cost;
  for (int k : h->active_ids) {
    const double w = h->mem[k].dp;
    cost.push_back({w * (h->mem[k].p_in + (h->mem[k].depth - 1) * w), k});
  }
  std::stable_sort(cost.begin(), cost.end(), [](const auto& x, const auto& y) { return x.first > y.first; });
  std::vector<double> load(h->ngroups, 0.0);
  for (const auto& ck : cost) {
    const int g = (int)(std::min_element(load.begin(), load.end()) - load.begin());
    load[g] += ck.first;
    h->group[g].push_back(ck.second);
  }
  for (auto& v : h->group) std::sort(v.begin(), v.end());
}

// The largest first-layer width p_in among the given members.
int max_pin(const pack_handle* h, const std::vector<int>& ids) {
  int m = 0;
  for (int k : ids) m = std::max(m, h->mem[k].p_in);
  return m;
}

// Rows per head-backward block: up to 256, dividing Bp.
int head_rows(const pack_handle* h) { return h->Bp % 256 == 0 ? 256 : h->Bp; }

// Shape of the Newton-Schulz iterate of member m's hidden weight l (1-based):
// padded [R x Cp] storage; X is [S x L], U or U^T (tall: true rows > true columns).
struct MuonShape {
  int R, Cp, S, L, r, c;
  bool tall;
};
MuonShape muon_shape(const pack_handle* h, const Member& m, int l) {
  MuonShape q;
  q.R = m.dp;
  q.Cp = l == 1 ? m.p_in : m.dp;
  q.r = m.width;
  q.c = l == 1 ? (m.d_emb ? h->cfg.d_in * m.d_emb : h->cfg.d_in) : m.width;
  q.tall = q.r > q.c;
  q.S = q.tall ? q.Cp : q.R;
  q.L = q.tall ? q.R : q.Cp;
  return q;
}

// Elements of one X buffer and of the A (or B') buffer for the given members.
template <typename It>
void muon_sizes(const pack_handle* h, It begin, It end, int64_t& xe, int64_t& ae) {
  xe = ae = 0;
  for (It it = begin; it != end; ++it) {
    const Member& m = h->mem[*it];
    for (int l = 1; l <= m.depth; ++l) {
      const MuonShape q = muon_shape(h, m, l);
      xe += round_up((int64_t)q.S * q.L, kChunk);
      ae += round_up((int64_t)q.S * q.S, kChunk);
    }
  }
}

// Tiles on and above the diagonal of a symmetric S x S result (the others are
// written as mirror images by the tiles above the diagonal).  Rows go in
// blocks as in add_tiles; within its row block a diagonal block takes small
// tiles on and above its own diagonal, and the columns right of it take the
// tile set's large tiles (a remainder of at most 128 columns small ones).
void add_tiles_sym(Plan& p, Launch& ln, int d, int S, int kdepth) {
  ln.ts = p.tile_set;
  auto push = [&](int m0, int n0, int shape) {
    const int tm = shape == kShapeSmall ? kSmallTile : kBigTile;
    const int tw = shape == kShapeBig ? kBigTile : kSmallTile;
    const int mb = std::min(tm, S - m0), nb = std::min(tw, S - n0);
    p.tiles.push_back(Tile{d, m0, n0, shape});
    // a tile above the diagonal also stores its mirror image
    p.cost.push_back((int64_t)kdepth * mb * nb * (m0 < n0 ? 2 : 1));
  };
  if (p.tile_set == TILES_SMALL) {
    for (int m0 = 0; m0 < S; m0 += kSmallTile)
      for (int n0 = m0; n0 < S; n0 += kSmallTile) push(m0, n0, kShapeSmall);
  } else {
    const bool big = p.tile_set == TILES_BIG;
    const int large = big ? kShapeBig : kShapeTall, tn = big ? kBigTile : kSmallTile;
    const int r = S % kBigTile;
    const int Mb = r == 0 ? S : (r > kSmallTile ? S - r + kBigTile : S - r);
    for (int m0 = 0; m0 < Mb; m0 += kBigTile) {
      const int e = std::min(m0 + kBigTile, S);  // end of the diagonal block
      for (int i0 = m0; i0 < e; i0 += kSmallTile)
        for (int n0 = i0; n0 < e; n0 += kSmallTile) push(i0, n0, kShapeSmall);
      const int rc = (S - e) % tn;
      const int Nb = big ? (rc == 0 || rc > kSmallTile ? S : S - rc) : S;
      for (int n0 = e; n0 < Nb; n0 += tn) push(m0, n0, large);
      for (int i0 = m0; i0 < e; i0 += kSmallTile)
        for (int n0 = Nb; n0 < S; n0 += kSmallTile) push(i0, n0, kShapeSmall);
    }
    for (int m0 = Mb; m0 < S; m0 += kSmallTile)
      for (int n0 = m0; n0 < S; n0 += kSmallTile) push(m0, n0, kShapeSmall);
  }
  ln.ntiles = (int)p.tiles.size() - ln.tile0;
}

void plan_muon(const pack_handle* h, const Bufs& bf, const std::vector<int> (&group)[kGroups], Plan& p) {
  const size_t es = h->elt();
  const TileSet saved = p.tile_set;
  p.tile_set = h->ns_tiles;
  int64_t xo = 0, ao = 0;
  struct Item {
    MuonShape q;
    int64_t xoff, aoff;
    int mi;  // its MuonMat in p.mmats
  };
  auto xp = [&](int par, int64_t off) { return (void*)(bf.mX[par] + (size_t)off * es); };
  auto ap = [&](const char* base, int64_t off) { return (void*)(base + (size_t)off * es); };
  p.mtile0.push_back(0);
  for (int hf = 0; hf < kGroups; ++hf) {
    p.mmat0[hf] = (int)p.mmats.size();
    p.mtileg[hf] = (int)p.mtiles.size();
    std::vector<Item> items;
    for (int k : group[hf]) {
      const Member& m = h->mem[k];
      for (int l = 1; l <= m.depth; ++l) {
        const MuonShape q = muon_shape(h, m, l);
        MuonMat mm{};
        mm.woff = m.toff[2 * (l - 1)];
        mm.xoff = xo;
        mm.aoff = ao;
        mm.R = q.R;
        mm.Cp = q.Cp;
        mm.tall = q.tall ? 1 : 0;
        mm.member = k;
        mm.decay = (float)(1.0 - m.muon_lr * m.wd);
        mm.step = (float)(m.muon_lr * std::sqrt(std::max(1.0, (double)q.r / q.c)));
        const int mi = (int)p.mmats.size();
        p.mmats.push_back(mm);
        for (int r0 = 0; r0 < q.R; r0 += 64)
          for (int c0 = 0; c0 < q.Cp; c0 += 64) p.mtiles.push_back(MuonTile{mi, r0, c0, 0});
        p.mtile0.push_back((int32_t)p.mtiles.size());
        items.push_back(Item{q, xo, ao, mi});
        xo += round_up((int64_t)q.S * q.L, kChunk);
        ao += round_up((int64_t)q.S * q.S, kChunk);
      }
    }
    // A = X X^T, one launch per parity of the X buffer it reads
    for (int par = 0; par < 2; ++par) {
      Launch& ln = p.nsA[par][hf];
      ln = Launch{(int)p.descs.size(), 0, (int)p.tiles.size(), 0, 0.0, 0.0};
      for (const Item& it : items) {
        GemmDesc d{};
        d.A = d.B = xp(par, it.xoff);
        d.lda = d.ldb = it.q.L;
        d.C = ap(bf.mA, it.aoff);
        d.ldc = it.q.S;
        d.M = d.N = it.q.S;
        d.Kd = it.q.L;
        add_tiles_sym(p, ln, (int)p.descs.size(), it.q.S, d.Kd);
        p.descs.push_back(d);
        ++ln.ndesc;
        const double s = std::min(it.q.r, it.q.c), l = std::max(it.q.r, it.q.c);
        ln.flops += s * (s + 1) * l;  // a symmetric result: the upper triangle
        ln.bytes += es * (s * l + s * s);
      }
      sort_launch(p, ln);
    }
    // B' = b A + c A A: A is stored exactly symmetric (mirrored tiles), so A A =
    // A A^T reads both operands depth-contiguous, and B' is symmetric too
    {
      Launch& ln = p.nsB[hf];
      ln = Launch{(int)p.descs.size(), 0, (int)p.tiles.size(), 0, 0.0, 0.0};
      for (const Item& it : items) {
        GemmDesc d{};
        d.A = d.B = ap(bf.mA, it.aoff);
        d.lda = d.ldb = it.q.S;
        d.C = ap(bf.mB, it.aoff);
        d.ldc = it.q.S;
        d.Y = ap(bf.mA, it.aoff);
        d.ldy = it.q.S;
        d.M = d.N = d.Kd = it.q.S;
        add_tiles_sym(p, ln, (int)p.descs.size(), it.q.S, d.Kd);
        p.descs.push_back(d);
        ++ln.ndesc;
        const double s = std::min(it.q.r, it.q.c);
        ln.flops += s * (s + 1) * s;  // a symmetric result: the upper triangle
        ln.bytes += es * 3.0 * s * s;
      }
      sort_launch(p, ln);
    }
    // X' = a X + B' X, reading X from buffer par and writing buffer 1 - par
    for (int par = 0; par < 2; ++par) {
      Launch& ln = p.nsX[par][hf];
      ln = Launch{(int)p.descs.size(), 0, (int)p.tiles.size(), 0, 0.0, 0.0};
      for (const Item& it : items) {
        GemmDesc d{};
        d.A = ap(bf.mB, it.aoff);
        d.lda = it.q.S;
        d.B = xp(par, it.xoff);
        d.ldb = it.q.L;
        d.C = xp(par ^ 1, it.xoff);
        d.ldc = it.q.L;
        d.Y = xp(par, it.xoff);
        d.ldy = it.q.L;
        d.M = it.q.S;
        d.N = it.q.L;
        d.Kd = it.q.S;
        // the weight the last iteration updates in its epilogue
        const MuonMat& mm = p.mmats[it.mi];
        d.poff = mm.woff;
        d.ns_tall = mm.tall;
        d.ns_decay = mm.decay;
        d.ns_step = mm.step;
        add_tiles(p, ln, (int)p.descs.size(), d.M, d.N, d.Kd);
        p.descs.push_back(d);
        ++ln.ndesc;
        const double s = std::min(it.q.r, it.q.c), l = std::max(it.q.r, it.q.c);
        ln.flops += 2.0 * s * s * l;
        ln.bytes += es * (s * s + 2.0 * s * l);
      }
      sort_launch(p, ln);
    }
  }
  p.mmat0[kGroups] = (int)p.mmats.size();
  p.mtileg[kGroups] = (int)p.mtiles.size();
  p.tile_set = saved;
}

// Tile set of one forward / data-gradient / weight-gradient launch whose
// 128 x 128 tiles number n_small: fixed by `forced` (>= 0), else 256 x 128 tiles
// when there are at least kTallMinTiles small ones (two full rounds of tall
// tiles at two workgroups per CU), small tiles otherwise.  Measured (ms per
// step, all small / all tall / chosen): 64 members of widths 64..2048 at batch
// 2048 (launches of 700..2800 small tiles) 6.29 / 5.76; 64 of widths
// 256..1024 at batch 1024 (500..840) 1.45 / 1.53 (tall dW alone 1.53);
// 32 of 256..1024 (~440) 0.63 / 0.67.
// Weight-gradient launches also need a depth (padded batch) of at least
// kTallMinDepthDw: their small tiles stream the fused optimizer over the whole
// staged gradient tile, which the tall tiles do not, and at a 1024-row batch
// that epilogue outweighs the tall tiles' faster main loop (the embedded first
// layer's dW: 7.05 ms small, 7.99 ms tall), at 2048 rows it does not
// (widths 64..2048: 6.29 -> 6.09 ms per step with tall dW tiles alone).
constexpr int kTallMinTiles = 1024, kTallMinDepthDw = 2048;
TileSet launch_tiles(const pack_handle* h, int forced, int64_t n_small, int min_depth = 0) {
  if (forced >= 0) return (TileSet)forced;
  if (h->prec != Prec::BF16 || h->Bp < min_depth) return TILES_SMALL;
  return n_small >= kTallMinTiles ? TILES_TALL : TILES_SMALL;
}
int64_t small_tiles(int M, int N) { return (int64_t)((M + kSmallTile - 1) / kSmallTile) * ((N + kSmallTile - 1) / kSmallTile); }

// Launch tables over the members of `group` (the active members split into
// streams; carve() sizes the workspace with every member in one group).
Plan build_plan(const pack_handle* h, const Bufs& bf, const std::vector<int> (&group)[kGroups],
                bool sizing = false) {
  Plan p;
  // sizing: small tiles for the main GEMMs (the largest tile count of any choice)
  auto choose = [&](int forced, int64_t n_small, int min_depth = 0) {
    return sizing ? TILES_SMALL : launch_tiles(h, forced, n_small, min_depth);
  };
  p.tile_set = h->tiles;
  const pack_config& c = h->cfg;
  const size_t es = h->elt();
  const void* wsrc = h->prec == Prec::BF16 ? (const void*)bf.shadow : (const void*)bf.theta;
  auto Hl = [&](int l) -> void* { return bf.H + (size_t)(l - 1) * h->A * es; };
  auto dzb = [&](int l) -> void* { return bf.dz + (size_t)(l & 1) * h->A * es; };
  auto wptr = [&](int k, int l) -> const void* {  // weight of hidden layer l (1-based) for GEMM reads
    return (const char*)wsrc + (size_t)h->mem[k].toff[2 * (l - 1)] * es;
  };
  auto act = [&](void* base, int k) -> void* { return (char*)base + (size_t)h->mem[k].act_off * es; };
  auto maskp = [&](int l, int k) -> uint32_t* {  // keep bits of H_l (1-based) of member k
    return bf.mask + (size_t)(l - 1) * (h->A / 32) + h->mem[k].act_off / 32;
  };
  auto h0 = [&](int k) -> void* { return bf.H0 + (size_t)h->mem[k].h0_off * es; };
  auto keepw = [&](int par, int l, int k) -> const uint32_t* {
    return bf.keepw + (size_t)par * c.L * (h->A / 32) + (maskp(l, k) - bf.mask);
  };
  for (int par = 0; par < 2; ++par)
  for (int hf = 0; hf < kGroups; ++hf)
  for (int l = 1; l <= c.L; ++l) {
    // forward: Z_l = H_{l-1} W_l^T + b_l, rows = batch (Bp), cols = dp; members
    // with fewer than l hidden blocks are not in the launch
    Launch f{(int)p.descs.size(), 0, (int)p.tiles.size(), 0, 0.0};
    int64_t nsm = 0;
    for (int k : group[hf])
      if (h->mem[k].depth >= l) nsm += small_tiles(h->Bp, h->mem[k].dp);
    // the embedded first layer (E produced in the GEMM): its own tile set
    p.tile_set = l == 1 && h->emb ? (sizing ? TILES_SMALL : h->emb_tiles) : choose(h->tiles_fwd, nsm);
    for (int k : group[hf]) {
      const Member& m = h->mem[k];
      if (m.depth < l) continue;
      ++f.ndesc;
      GemmDesc d{};
      d.A = l == 1 ? (m.d_emb ? nullptr : h0(k)) : act(Hl(l - 1), k);  // the embedded E is produced in the GEMM
      d.lda = l == 1 ? m.p_in : m.dp;
      d.B = wptr(k, l);
      d.ldb = l == 1 ? m.p_in : m.dp;
      d.C = act(Hl(l), k);
      d.ldc = m.dp;
      d.bias = bf.theta + m.toff[2 * (l - 1) + 1];
      d.M = h->Bp;
      d.N = m.dp;
      d.Kd = l == 1 ? m.p_in : m.dp;
      d.width = m.width;
      d.member = k;
      d.drop_t = m.t;
      d.drop_s = (float)m.scale;
      d.mask = maskp(l, k);
      d.keepw = keepw(par, l, k);
      if (l == 1 && h->stream_rows && m.d_emb == 0 && !sizing) {  // rows straight from the data copy
        d.A = h->xb;
        d.lda = h->Pin;
        d.xrows = bf.idx_ok + (size_t)k * c.B;
        d.xrows_n = c.B;
        d.xsrc_rows = h->data_N;
      }
      add_tiles(p, f, (int)p.descs.size(), h->Bp, m.dp, d.Kd);
      p.descs.push_back(d);
      {
        const double fi = l == 1 ? (m.d_emb ? (double)c.d_in * m.d_emb : c.d_in) : m.width, w = m.width;
        f.flops += 2.0 * c.B * w * fi;
        // H_{l-1} and W_l read, H_l written (2-byte elements in bf16), keep words read, mask words written;
        // the embedded first layer reads the batch's data rows and the column table instead of E
        f.bytes += (double)h->elt() * (fi * w + c.B * w) + c.B * w / 4.0 +
                   (l == 1 && m.d_emb ? 4.0 * c.B * c.d_in + 16.0 * fi : (double)h->elt() * c.B * fi);
      }
    }
    sort_launch(p, f);
    p.fwd[par][hf].push_back(f);
  }
  {
    // evaluation, layer 1: every member reads the same validation rows (H_0 block 0)
    Launch f{(int)p.descs.size(), 0, (int)p.tiles.size(), 0, 0.0};
    int64_t nsm = 0;
    for (int hf = 0; hf < kGroups; ++hf) {
      f.ndesc += (int)group[hf].size();
      for (int k : group[hf]) nsm += small_tiles(h->Bp, h->mem[k].dp);
    }
    p.tile_set = h->emb ? (sizing ? TILES_SMALL : h->emb_tiles) : choose(h->tiles_fwd, nsm);
    for (int hf = 0; hf < kGroups; ++hf)
      for (int i = 0; i < (int)group[hf].size(); ++i) {
        const int k = group[hf][i];
        GemmDesc d = p.descs[p.fwd[0][hf][0].desc0 + i];
        if (h->mem[k].d_emb == 0) d.A = h0(0);  // embedded members read their own E block
        d.xrows = nullptr;                      // evaluation reads the gathered validation rows
        add_tiles(p, f, (int)p.descs.size(), h->Bp, h->mem[k].dp, d.Kd);
        p.descs.push_back(d);
      }
    sort_launch(p, f);
    p.fwd1_eval = f;
  }
  for (int hf = 0; hf < kGroups; ++hf)
  for (int l = 1; l <= c.L; ++l) {
    // weight gradient: dW_l^T[out, in] = sum_rows dZ_l[row, out] H_{l-1}[row, in]
    Launch w{(int)p.descs.size(), 0, (int)p.tiles.size(), 0, 0.0};
    int64_t nsm = 0;
    for (int k : group[hf])
      if (h->mem[k].depth >= l) nsm += small_tiles(h->mem[k].dp, l == 1 ? h->mem[k].p_in : h->mem[k].dp);
    p.tile_set = l == 1 && h->emb ? TILES_SMALL : choose(h->tiles_dw, nsm, kTallMinDepthDw);
    for (int k : group[hf]) {
      const Member& m = h->mem[k];
      if (m.depth < l) continue;
      ++w.ndesc;
      GemmDesc d{};
      d.A = act(dzb(l), k);
      d.lda = m.dp;
      d.B = l == 1 ? (m.d_emb ? nullptr : h0(k)) : act(Hl(l - 1), k);
      d.ldb = l == 1 ? m.p_in : m.dp;
      d.C = bf.grad + m.toff[2 * (l - 1)];
      d.ldc = l == 1 ? m.p_in : m.dp;
      d.M = m.dp;
      d.N = l == 1 ? m.p_in : m.dp;
      d.Kd = h->Bp;
      d.member = k;
      d.poff = m.toff[2 * (l - 1)];
      d.lr = (float)m.lr;
      d.wd = (float)m.wd;
      // the rows that exist (the member's true width): the optimizer leaves the zero padding rows
      // alone (1.365 -> 1.359 ms per step; skipping the padding columns as well, which leaves
      // holes in the rows' streaming stores, measured 1.362 ms, and 12.5 against 12.2 ms on the
      // embedded step)
      d.opt_rows = m.width;
      if (l == 1 && h->stream_rows && m.d_emb == 0 && !sizing) {  // rows straight from the data copy
        d.B = h->xb;
        d.ldb = h->Pin;
        d.xrows = bf.idx_ok + (size_t)k * c.B;
        d.xrows_n = c.B;
        d.xsrc_rows = h->data_N;
      }
      if (l == 1 && m.d_emb) {  // E produced in the GEMM from the batch rows' data rows
        d.xrows = bf.idx_ok + (size_t)k * c.B;
        d.xrows_n = c.B;
      }
      add_tiles(p, w, (int)p.descs.size(), d.M, d.N, d.Kd);
      p.descs.push_back(d);
      {
        const double fi = l == 1 ? (m.d_emb ? (double)c.d_in * m.d_emb : c.d_in) : m.width, wd = m.width;
        w.flops += 2.0 * c.B * wd * fi;
        // dZ_l and H_{l-1} read (the embedded first layer: the data rows and the column table);
        // per weight: the fused AdamW's theta, m, v read and written (24 B) and the bf16 shadow
        // written (2 B), plus the fp32 gradient when it is kept
        w.bytes += (double)h->elt() * c.B * wd +
                   (l == 1 && m.d_emb ? 4.0 * c.B * c.d_in + 16.0 * fi : (double)h->elt() * c.B * fi) +
                   wd * fi * (24.0 + (h->prec == Prec::BF16 ? 2.0 : 0.0) + (c.keep_grads ? 4.0 : 0.0));
      }
    }
    sort_launch(p, w);
    p.dw[hf].push_back(w);
    // data gradient (l >= 2): dZ_{l-1} = (dZ_l W_l) * [H_{l-1} > 0] * s_k
    Launch x{(int)p.descs.size(), 0, (int)p.tiles.size(), 0, 0.0};
    if (l >= 2) {
      int64_t nsx = 0;
      for (int k : group[hf])
        if (h->mem[k].depth >= l) nsx += small_tiles(h->Bp, h->mem[k].dp);
      p.tile_set = choose(h->tiles_dx, nsx);
      for (int k : group[hf]) {
        const Member& m = h->mem[k];
        if (m.depth < l) continue;
        ++x.ndesc;
        GemmDesc d{};
        d.A = act(dzb(l), k);
        d.lda = m.dp;
        d.B = wptr(k, l);
        d.ldb = m.dp;
        d.C = act(dzb(l - 1), k);
        d.mask = maskp(l - 1, k);
        d.colpart = bf.colpart + (size_t)(l - 2) * (h->A / kPartRows) + h->mem[k].act_off / kPartRows;
        d.ldc = m.dp;
        d.M = h->Bp;
        d.N = m.dp;
        d.Kd = m.dp;
        d.member = k;
        d.drop_s = (float)m.scale;
        add_tiles(p, x, (int)p.descs.size(), h->Bp, m.dp, d.Kd);
        p.descs.push_back(d);
        x.flops += 2.0 * c.B * m.width * m.width;
        // dZ_l and W_l read, dZ_{l-1} written, mask words read, bias partials written
        x.bytes += (double)h->elt() * (2.0 * c.B * m.width + (double)m.width * m.width) + c.B * m.width / 8.0 +
                   4.0 * (h->Bp / kPartRows) * m.width;
      }
      sort_launch(p, x);
    }
    p.dx[hf].push_back(x);
  }
  // gradient-sum work items of group g (one launch after the group's last
  // backward launch): coltiles[sumtile0[g] .. sumtile0[g + 1]) -- the bias
  // columns of every dX launch (layer l >= 2: b_{l-1} of the members with at
  // least l hidden blocks), then every member's head columns, then one loss
  // item per member
  for (int hf = 0; hf < kGroups; ++hf) {
    p.sumtile0[hf] = (int)p.coltiles.size();
    for (int l = 2; l <= c.L; ++l)
      for (int k : group[hf])
        if (h->mem[k].depth >= l)
          for (int c0 = 0; c0 < h->mem[k].dp; c0 += 64) p.coltiles.push_back(ColTile{k, c0, l - 2});
    for (int k : group[hf])
      for (int c0 = 0; c0 < h->mem[k].dp; c0 += 64) p.coltiles.push_back(ColTile{k, c0, kSumHead});
    for (int k : group[hf]) p.coltiles.push_back(ColTile{k, 0, kSumLoss});
  }
  p.sumtile0[kGroups] = (int)p.coltiles.size();
  const TileSet saved_ts = p.tile_set;
  p.tile_set = TILES_SMALL;  // the embedding's data-gradient GEMM runs small tiles only
  for (int hf = 0; hf < kGroups; ++hf) {
    Launch& ln = p.de[hf];
    ln = Launch{(int)p.descs.size(), 0, (int)p.tiles.size(), 0, 0.0, 0.0};
    for (int k : group[hf]) {
      const Member& m = h->mem[k];
      if (!m.d_emb) continue;
      GemmDesc d{};
      d.A = act(dzb(1), k);
      d.lda = m.dp;
      d.B = wptr(k, 1);  // W_1 [dp, p_in] read as rows-contiguous: element (n, k) at W_1[k * p_in + n]
      d.ldb = m.p_in;
      d.C = bf.dE + m.h0_off / 16;
      d.ldc = m.p_in;
      d.M = h->Bp;
      d.N = m.p_in;
      d.Kd = m.dp;
      d.member = k;
      add_tiles(p, ln, (int)p.descs.size(), d.M, d.N, d.Kd);
      p.descs.push_back(d);
      ++ln.ndesc;
      const double e = (double)c.d_in * m.d_emb;
      ln.flops += 2.0 * c.B * m.width * e;
      // dZ_1 and W_1 read, x of the rows' features, four fp32 sums per column and 64-row block
      ln.bytes += (double)h->elt() * (c.B * m.width + m.width * e) + 4.0 * c.B * c.d_in + 16.0 * (h->Bp / 64) * e;
    }
    sort_launch(p, ln);
  }
  p.tile_set = saved_ts;
  const int hcols = head_bwd_cols(c.d_out), hrb = head_rows(h);
  for (int hf = 0; hf < kGroups; ++hf) {
    p.headtile0[hf] = (int)p.headtiles.size();
    p.member0[hf] = (int)p.members.size();
    for (int r0 = 0; r0 < h->Bp; r0 += hrb)
      for (int k : group[hf])
        for (int c0 = 0; c0 < h->mem[k].dp; c0 += hcols) p.headtiles.push_back(HeadTile{k, c0, r0});
    for (int k : group[hf]) p.members.push_back(k);
  }
  p.headtile0[kGroups] = (int)p.headtiles.size();
  p.member0[kGroups] = (int)p.members.size();
  if (h->muon) plan_muon(h, bf, group, p);
  return p;
}

struct Carve {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t count) {
    off = (size_t)round_up((int64_t)off, 256);
    T* p = reinterpret_cast<T*>(reinterpret_cast<uintptr_t>(base) + off);
    off += count * sizeof(T);
    return p;
  }
};

// Lays out the workspace.  With base == nullptr it only measures: the
// pointers are then offsets from address 0 and are never dereferenced.
size_t carve(const pack_handle* h, char* base, Bufs& bf) {
  const pack_config& c = h->cfg;
  Carve cv{base};
  bf.theta = cv.take<float>(h->P);
  bf.grad = cv.take<float>(h->P);
  bf.m = cv.take<float>(h->P);
  bf.v = cv.take<float>(h->P);
  bf.shadow = h->prec == Prec::BF16 ? cv.take<uint16_t>(h->P) : nullptr;
  // embedded packs never store E (the first layer's GEMMs produce it)
  bf.H0 = h->emb ? nullptr : cv.take<char>((size_t)h->H0e * h->elt());
  // each member's sums at its E offset / 16 (Bp is a multiple of 256, so the
  // offsets divide; a member's [Bp / 64][4][p_in] sums fill Bp p_in / 16)
  bf.dE = h->emb ? cv.take<float>((size_t)h->H0e / 16) : nullptr;
  bf.etab = h->emb ? cv.take<float4>((size_t)h->Etab) : nullptr;
  bf.H = cv.take<char>((size_t)c.L * h->A * h->elt());
  bf.dz = cv.take<char>((size_t)2 * h->A * h->elt());
  bf.colpart = cv.take<float>((size_t)std::max(1, c.L - 1) * (h->A / kPartRows));
  bf.mask = cv.take<uint32_t>((size_t)c.L * (h->A / 32));
  bf.keepw = cv.take<uint32_t>((size_t)2 * c.L * (h->A / 32));
  bf.zeros = cv.take<char>(256);
  bf.dY = cv.take<float>((size_t)c.K * h->Bp * c.d_out);
  bf.rowloss = cv.take<float>((size_t)c.K * h->Bp);
  bf.d_mem = cv.take<MemberDev>(c.K);
  bf.d_chunks = cv.take<uint32_t>(h->chunk_tab.size());
  bf.d_aux = cv.take<uint32_t>(h->aux_chunks.size());
  bf.d_bias_off = cv.take<int64_t>((size_t)c.L * c.K);
  std::vector<int> all[kGroups];
  for (int k = 0; k < c.K; ++k) all[0].push_back(k);
  if (h->muon) {
    int64_t xe = 0, ae = 0;
    muon_sizes(h, all[0].begin(), all[0].end(), xe, ae);
    bf.mX[0] = cv.take<char>((size_t)xe * h->elt());
    bf.mX[1] = cv.take<char>((size_t)xe * h->elt());
    bf.mA = cv.take<char>((size_t)ae * h->elt());
    bf.mB = cv.take<char>((size_t)ae * h->elt());
  }
  // The tables are sized by a plan with every member in one launch per layer
  // and small tiles for the main GEMMs: any tile set, and any split of the
  // members, takes at most as many tiles.
  Plan plan = build_plan(h, bf, all, true);
  bf.tile_cap = plan.tiles.size();
  if (h->muon) {
    bf.mpart = cv.take<double>(plan.mtiles.size());
    bf.minv = cv.take<float>(plan.mmats.size());
    bf.d_mmats = cv.take<MuonMat>(plan.mmats.size());
    bf.d_mtiles = cv.take<MuonTile>(plan.mtiles.size());
    bf.d_mtile0 = cv.take<int32_t>(plan.mtile0.size());
  }
  bf.d_descs = cv.take<GemmDesc>(plan.descs.size());
  bf.d_tiles = cv.take<Tile>(plan.tiles.size());
  bf.d_coltiles = cv.take<ColTile>(plan.coltiles.size());
  bf.d_headtiles = cv.take<HeadTile>(plan.headtiles.size());
  bf.d_members = cv.take<int32_t>(plan.members.size());
  bf.d_active = cv.take<int32_t>(c.K);
  bf.headpart = cv.take<float>((size_t)(h->Bp / head_rows(h)) * (c.d_out + 1) * (h->A / h->Bp));
  bf.idx_ok = cv.take<int32_t>((size_t)c.K * c.B);
  bf.status = cv.take<uint32_t>(64);
  return (size_t)round_up((int64_t)cv.off, 256);
}

int check_member(const pack_handle* h, int32_t k) {
  if (!h) return fail(PACK_EINVAL, "handle is NULL");
  if (k < 0 || k >= h->cfg.K) return fail(PACK_EINVAL, "member %d out of [0, %d)", k, h->cfg.K);
  return PACK_OK;
}

uint32_t as_u32(uint64_t x) { return (uint32_t)(x & 0xFFFFFFFFu); }

GemmArgs base_args(const pack_handle* h) {
  GemmArgs a{};
  a.descs = h->b.d_descs;
  a.tiles = h->b.d_tiles;
  a.zeros = h->b.zeros;
  a.tile_set = h->tiles;
  const Key kd = stream_key(h->cfg.seed, kTagDropout);
  a.key0 = kd.k0;
  a.key1 = kd.k1;
  return a;
}

GemmArgs for_launch(GemmArgs a, const Launch& ln) {
  a.tiles += ln.tile0;
  a.ntiles = ln.ntiles;
  a.tile_set = ln.ts;
  return a;
}

// The first-layer arguments of a GEMM that produces the embedded input E
// (OP_EMB): the data X (N rows), and the batch indices (training forward) or
// the first data row (idx == nullptr: evaluation).
void set_emb(const pack_handle* h, GemmArgs& a, const float* X, int64_t N, const int32_t* idx, int64_t row_base) {
  a.emb_x = X;
  a.emb_x_rows = N;
  a.emb_idx = idx;
  a.emb_row_base = row_base;
  a.emb_mem = h->b.d_mem;
  a.emb_d_in = h->cfg.d_in;
  a.emb_tab = h->b.etab;
}

hipEvent_t pool_event(pack_handle* h) {
  if (h->pool_used == h->event_pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    h->event_pool.push_back(e);
  }
  return h->event_pool[h->pool_used++];
}

int group_id(pack_handle* h, const std::string& name, int kind) {
  for (size_t i = 0; i < h->groups.size(); ++i)
    if (h->groups[i].name == name) return (int)i;
  h->groups.push_back(ProfGroup{name, kind});
  return (int)h->groups.size() - 1;
}

// Runs `fn` (which enqueues one kernel on `stream`) and, when profiling,
// brackets it with events and attributes `work` to the named kernel.
template <typename F>
hipError_t timed(pack_handle* h, const char* name, int kind, double flops, double bytes, hipStream_t stream, F fn) {
  if (!h->prof) return fn();
  hipEvent_t a = pool_event(h), b = pool_event(h);
  if (!a || !b) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(a, stream);
  if (e != hipSuccess) return e;
  e = fn();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, stream);
  const int g = group_id(h, name, kind);
  h->groups[g].flops += flops;  // summed here, averaged per launch when read
  h->groups[g].bytes += bytes;
  h->timed.push_back(TimedLaunch{g, a, b});
  return e;
}

// The column tables of the listed members' embeddings from their current
// parameters (d_members: the same member ids in device memory).
hipError_t emb_tables(pack_handle* h, const int32_t* d_members, const std::vector<int>& ids, hipStream_t s) {
  double nb = 0;
  for (int k : ids) nb += 32.0 * h->mem[k].p_in;  // four parameters read, one 16-byte entry written per column
  return timed(h, "embed_table", 1, 0.0, nb, s, [&] {
    return launch_embed_table(h->prec, h->cfg.d_in, h->b.d_mem, d_members, (int)ids.size(), max_pin(h, ids),
                              h->b.theta, h->b.etab, s);
  });
}

void set_active_ids(pack_handle* h) {
  h->active_ids.clear();
  for (int k = 0; k < h->cfg.K; ++k)
    if (h->active[k]) h->active_ids.push_back(k);
}

// Builds the launch tables of the active members, uploads them (and the AdamW
// list of the active members' biases and heads) into the bound workspace, and
// records the launches.  Synchronizes `stream`: the host tables are freed on
// return.  The caller's earlier work on `stream` is ordered before the copies.
int upload_plan(pack_handle* h, hipStream_t stream) {
  const pack_config& c = h->cfg;
  Plan plan = build_plan(h, h->b, h->group);
  if (plan.tiles.size() > h->b.tile_cap)
    return fail(PACK_EINVAL, "internal: the plan holds %zu GEMM tiles, the device table %zu", plan.tiles.size(),
                h->b.tile_cap);
  std::vector<uint32_t> aux;
  for (uint32_t ch : h->aux_chunks)
    if (h->active[h->chunk_tab[ch] & 0x7FFFFFFFu]) aux.push_back(ch);
  h->n_aux_active = (int64_t)aux.size();
  auto up = [&](void* dst, const void* src, size_t bytes) {
    return bytes ? hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, stream) : hipSuccess;
  };
  HIP_TRY(up(h->b.d_aux, aux.data(), aux.size() * 4));
  HIP_TRY(up(h->b.d_active, h->active_ids.data(), h->active_ids.size() * 4));
  HIP_TRY(up(h->b.d_descs, plan.descs.data(), plan.descs.size() * sizeof(GemmDesc)));
  HIP_TRY(up(h->b.d_tiles, plan.tiles.data(), plan.tiles.size() * sizeof(Tile)));
  HIP_TRY(up(h->b.d_coltiles, plan.coltiles.data(), plan.coltiles.size() * sizeof(ColTile)));
  HIP_TRY(up(h->b.d_headtiles, plan.headtiles.data(), plan.headtiles.size() * sizeof(HeadTile)));
  HIP_TRY(up(h->b.d_members, plan.members.data(), plan.members.size() * sizeof(int32_t)));
  if (h->muon) {
    HIP_TRY(up(h->b.d_mmats, plan.mmats.data(), plan.mmats.size() * sizeof(MuonMat)));
    HIP_TRY(up(h->b.d_mtiles, plan.mtiles.data(), plan.mtiles.size() * sizeof(MuonTile)));
    HIP_TRY(up(h->b.d_mtile0, plan.mtile0.data(), plan.mtile0.size() * sizeof(int32_t)));
  }
  HIP_TRY(hipStreamSynchronize(stream));
  h->n_mmats = (int)plan.mmats.size();
  h->n_mtiles = (int)plan.mtiles.size();
  for (int g = 0; g <= kGroups; ++g) {
    h->mmat0[g] = plan.mmat0[g];
    h->mtileg[g] = plan.mtileg[g];
  }
  for (int g = 0; g < kGroups; ++g) {
    for (int par = 0; par < 2; ++par) {
      h->nsA[par][g] = plan.nsA[par][g];
      h->nsX[par][g] = plan.nsX[par][g];
    }
    h->nsB[g] = plan.nsB[g];
  }
  for (int hf = 0; hf < kGroups; ++hf) h->de[hf] = plan.de[hf];
  for (int hf = 0; hf < kGroups; ++hf) {
    h->fwd[0][hf] = plan.fwd[0][hf];
    h->fwd[1][hf] = plan.fwd[1][hf];
    h->dx[hf] = plan.dx[hf];
    h->dw[hf] = plan.dw[hf];
  }
  h->fwd1_eval = plan.fwd1_eval;
  for (int g = 0; g <= kGroups; ++g) h->sumtile0[g] = plan.sumtile0[g];
  for (int i = 0; i <= kGroups; ++i) {
    h->headtile0[i] = plan.headtile0[i];
    h->member0[i] = plan.member0[i];
  }
  h->ncoltiles = (int)plan.coltiles.size();
  h->nheadtiles = (int)plan.headtiles.size();
  h->head_rb = head_rows(h);
  (void)c;
  return PACK_OK;
}

const char* gemm_name(Prec p, OpKind a, OpKind b, EpiKind e);

// Muon step of the hidden weights of member group g's active members (their
// gradients are in grad): momentum and tile norms, inverse norms, X0, ns_steps
// Newton-Schulz iterations of three grouped GEMMs, update.  On the group's
// stream after its backward pass, so one group's step overlaps the others'
// backward passes and Muon steps.
hipError_t muon_step(pack_handle* h, const GemmArgs& base, int g, hipStream_t stream) {
  const int mat0 = h->mmat0[g], nmats = h->mmat0[g + 1] - mat0;
  const int tile0 = h->mtileg[g], ntiles = h->mtileg[g + 1] - tile0;
  if (nmats == 0) return hipSuccess;
  const pack_config& c = h->cfg;
  const float mu = (float)c.muon_momentum;
  const int nest = c.muon_nesterov ? 1 : 0;
  const MuonTile* tiles = h->b.d_mtiles + tile0;
  const double wbytes = (double)ntiles * 64 * 64;  // upper bound of the weights' elements
  hipError_t e = timed(h, "muon_prep", 1, 0.0, wbytes * 12.0, stream, [&] {
    return launch_muon_prep(h->b.d_mmats, tiles, ntiles, h->b.grad, h->b.m, mu, nest, h->b.mpart + tile0, stream);
  });
  if (e != hipSuccess) return e;
  e = timed(h, "muon_norm", 1, 0.0, 8.0 * ntiles, stream, [&] {
    return launch_muon_norm(h->b.d_mtile0 + mat0, nmats, h->b.mpart, h->b.minv + mat0, stream);
  });
  if (e != hipSuccess) return e;
  e = timed(h, "muon_convert", 1, 0.0, wbytes * (8.0 + h->elt()), stream, [&] {
    return launch_muon_convert(h->prec, h->b.d_mmats, tiles, ntiles, h->b.grad, h->b.m, mu, nest, h->b.minv,
                               h->b.mX[0], stream);
  });
  if (e != hipSuccess) return e;
  static const float kA = 3.4445f, kB = -4.7750f, kC = 2.0315f;
  auto ns_args = [&](const GemmArgs& b0, const Launch& ln, OpKind bk, float alpha, float beta, bool sym) {
    GemmArgs ga = b0;
    ga.tiles += ln.tile0;
    ga.ntiles = ln.ntiles;
    ga.tile_set = h->ns_tiles;
    ga.ns_alpha = alpha;
    ga.ns_beta = beta;
    ga.ns_sym = sym ? 1 : 0;
    return timed(h, gemm_name(h->prec, OP_KMAJ, bk, EPI_NS), 0, ln.flops, ln.bytes, stream,
                 [&] { return launch_gemm(h->prec, OP_KMAJ, bk, EPI_NS, ga, stream); });
  };
  auto ns = [&](const Launch& ln, OpKind bk, float alpha, float beta, bool sym) {
    return ns_args(base, ln, bk, alpha, beta, sym);
  };
  // the last iteration's X launch applies the update in its epilogue
  // (TABPACK_MUON_FUSED_UPDATE=0: a separate update kernel reads the stored X)
  const bool fused = h->muon_fused;
  for (int it = 0; it < h->ns_steps; ++it) {
    const int par = it & 1;
    if ((e = ns(h->nsA[par][g], OP_KMAJ, 0.0f, 1.0f, true)) != hipSuccess) return e;
    if ((e = ns(h->nsB[g], OP_KMAJ, kB, kC, true)) != hipSuccess) return e;
    if (fused && it + 1 == h->ns_steps) {
      GemmArgs fa = base;
      fa.ns_theta = h->b.theta;
      fa.ns_shadow = h->b.shadow;
      if ((e = ns_args(fa, h->nsX[par][g], OP_RMAJ, kA, 1.0f, false)) != hipSuccess) return e;
      return hipSuccess;
    }
    if ((e = ns(h->nsX[par][g], OP_RMAJ, kA, 1.0f, false)) != hipSuccess) return e;
  }
  return timed(h, "muon_update", 1, 0.0, wbytes * (8.0 + h->elt() + (h->prec == Prec::BF16 ? 2.0 : 0.0)), stream,
               [&] {
                 return launch_muon_update(h->prec, h->b.d_mmats, tiles, ntiles, h->b.theta, h->b.shadow,
                                           h->b.mX[h->ns_steps & 1], stream);
               });
}

const char* gemm_name(Prec p, OpKind a, OpKind b, EpiKind e) {
  static const char* ops[] = {"kmaj", "rmaj", "emb"};
  static const char* epis[] = {"fwd", "fwd_eval", "dx", "dw", "ns", "de"};
  static thread_local char buf[64];
  snprintf(buf, sizeof buf, "gemm_%s_%s_%s_%s", p == Prec::BF16 ? "bf16" : "f32", ops[a], ops[b], epis[e]);
  return buf;
}

}  // namespace

extern "C" {

const char* pack_last_error(void) { return g_err.c_str(); }

int pack_init(const pack_config* cfg, pack_handle** out) {
  if (!out) return fail(PACK_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = validate(cfg);
  if (rc) return rc;
  pack_handle* h = new (std::nothrow) pack_handle();
  if (!h) return fail(PACK_EINVAL, "out of host memory");
  h->cfg = *cfg;
  h->cfg.members = nullptr;
  h->prec = cfg->precision == PACK_PREC_BF16 ? Prec::BF16 : Prec::FP32;
  h->task = (Task)cfg->task;
  h->q = cfg->quantum ? cfg->quantum : 32;
  // The tile sets of the main GEMMs are chosen per launch (launch_tiles);
  // TABPACK_GEMM_TILES=big|tall|small fixes them all, TABPACK_TILES_FWD / _DX /
  // _DW one kind.  h->tiles: the set of the remaining bf16 GEMM launches.
  h->tiles = TILES_SMALL;
  if (const char* e = getenv("TABPACK_GEMM_TILES")) {
    const std::string v(e);
    h->tiles = v == "big" ? TILES_BIG : (v == "tall" ? TILES_TALL : TILES_SMALL);
  }
  if (h->prec == Prec::FP32) h->tiles = TILES_SMALL;
  auto tile_env = [&](const char* name) {
    const char* e = getenv(name);
    if (h->prec == Prec::FP32) return (int)TILES_SMALL;
    if (!e) e = getenv("TABPACK_GEMM_TILES");
    if (!e) return -1;
    const std::string v(e);
    return (int)(v == "big" ? TILES_BIG : (v == "tall" ? TILES_TALL : TILES_SMALL));
  };
  h->tiles_fwd = tile_env("TABPACK_TILES_FWD");
  h->tiles_dx = tile_env("TABPACK_TILES_DX");
  h->tiles_dw = tile_env("TABPACK_TILES_DW");
  // Newton-Schulz GEMMs: small tiles measured 3.79 ms per Muon step on the
  // 64-member regression workload, tall 4.03, big 5.53; TABPACK_NS_TILES overrides
  h->ns_tiles = TILES_SMALL;
  if (const char* e = getenv("TABPACK_NS_TILES")) {
    const std::string v(e);
    h->ns_tiles = v == "big" ? TILES_BIG : (v == "tall" ? TILES_TALL : TILES_SMALL);
  }
  if (h->prec == Prec::FP32) h->ns_tiles = TILES_SMALL;
  // the embedded first layer's forward: wide tiles in bf16 (each produced E
  // element feeds 256 output columns); TABPACK_EMB_TILES=small overrides
  h->emb_tiles = h->prec == Prec::BF16 ? TILES_WIDE : TILES_SMALL;
  if (const char* e = getenv("TABPACK_EMB_TILES"))
    if (std::string(e) == "small") h->emb_tiles = TILES_SMALL;
  if (const char* e = getenv("TABPACK_MUON_FUSED_UPDATE")) h->muon_fused = std::string(e) != "0";
  h->muon = cfg->optimizer == PACK_OPT_MUON;
  h->emb = cfg->emb_lo > 0;
  h->ns_steps = cfg->ns_steps ? cfg->ns_steps : 5;
  h->Bp = (int)round_up(cfg->B, kRowAlign);
  h->Pin = (int)round_up(cfg->d_in, 8);
  h->mem.resize(cfg->K);
  if (cfg->members) {
    for (int k = 0; k < cfg->K; ++k) {
      const pack_member_hp& e = cfg->members[k];
      if (e.width < 1 || e.width > 16384 || !(e.dropout >= 0 && e.dropout < 1) || !(e.lr > 0) ||
          !(e.wd >= 0) || e.depth < 0 || e.depth > cfg->L ||
          (cfg->optimizer == PACK_OPT_MUON && !(e.muon_lr > 0)) ||
          (cfg->emb_lo > 0 && (e.d_emb < 8 || e.d_emb > 32 || !(e.sigma > 0)))) {
        delete h;
        return fail(PACK_EINVAL, "explicit hyperparameters of member %d out of range", k);
      }
      h->mem[k].width = e.width;
      h->mem[k].dropout = e.dropout;
      h->mem[k].lr = e.lr;
      h->mem[k].wd = e.wd;
      h->mem[k].depth = e.depth ? e.depth : cfg->L;
      h->mem[k].muon_lr = cfg->optimizer == PACK_OPT_MUON ? e.muon_lr : 0.0;
      h->mem[k].d_emb = cfg->emb_lo > 0 ? e.d_emb : 0;
      h->mem[k].sigma = cfg->emb_lo > 0 ? e.sigma : 0.0;
    }
  } else {
    sample_members(h);
  }
  for (Member& m : h->mem) {
    m.t = (uint32_t)std::min(std::floor(m.dropout * 65536.0), 65535.0);  // threshold of a 16-bit draw
    m.scale = 1.0 / (1.0 - m.dropout);
  }
  plan_layout(h);
  h->active.assign(cfg->K, 1);
  set_active_ids(h);
  split_members(h);
  init_params(h);
  *out = h;
  g_err.clear();
  return PACK_OK;
}

int pack_destroy(pack_handle* h) {
  if (h) {
    for (hipEvent_t e : h->event_pool) (void)hipEventDestroy(e);
    if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
    if (h->ev_join) (void)hipEventDestroy(h->ev_join);
    for (hipEvent_t e : h->ev_keep)
      if (e) (void)hipEventDestroy(e);
    if (h->side) (void)hipStreamDestroy(h->side);
    if (h->ev_split) (void)hipEventDestroy(h->ev_split);
    for (int g = 1; g < kGroups; ++g) {
      if (h->ev_merge[g]) (void)hipEventDestroy(h->ev_merge[g]);
      if (h->gstream[g]) (void)hipStreamDestroy(h->gstream[g]);
    }
    for (hipEvent_t e : h->ev_gather)
      if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : h->ev_bias)
      if (e) (void)hipEventDestroy(e);
  }
  delete h;
  return PACK_OK;
}

int pack_get_hparams(const pack_handle* h, pack_member_hp* out) {
  if (!h || !out) return fail(PACK_EINVAL, "NULL argument");
  for (int k = 0; k < h->cfg.K; ++k) {
    const Member& m = h->mem[k];
    out[k] = pack_member_hp{m.width, m.dp, m.t, m.depth, m.dropout, m.lr, m.wd, m.scale, m.muon_lr, m.d_emb, 0,
                            m.sigma};
  }
  return PACK_OK;
}

int pack_workspace_size(const pack_handle* h, size_t* bytes) {
  if (!h || !bytes) return fail(PACK_EINVAL, "NULL argument");
  Bufs tmp;
  *bytes = carve(h, nullptr, tmp);
  return PACK_OK;
}

int pack_bind(pack_handle* h, void* workspace, size_t bytes, hipStream_t stream) {
  if (!h || !workspace) return fail(PACK_EINVAL, "NULL argument");
  if (reinterpret_cast<uintptr_t>(workspace) % 256) return fail(PACK_EINVAL, "workspace must be 256-byte aligned");
  size_t need = 0;
  pack_workspace_size(h, &need);
  if (bytes < need) return fail(PACK_EINVAL, "workspace has %zu bytes, %zu needed", bytes, need);
  carve(h, static_cast<char*>(workspace), h->b);
  if (!h->side) {
    HIP_TRY(hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking));
    HIP_TRY(hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&h->ev_join, hipEventDisableTiming));
    for (hipEvent_t& e : h->ev_keep) HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&h->ev_split, hipEventDisableTiming));
    for (int g = 1; g < kGroups; ++g) {
      HIP_TRY(hipStreamCreateWithFlags(&h->gstream[g], hipStreamNonBlocking));
      HIP_TRY(hipEventCreateWithFlags(&h->ev_merge[g], hipEventDisableTiming));
    }
    for (hipEvent_t& e : h->ev_gather) HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    for (hipEvent_t& e : h->ev_bias) HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }
  h->keep_ready = 0;
  HIP_TRY(hipMemsetAsync(workspace, 0, need, stream));
  HIP_TRY(hipMemcpyAsync(h->b.theta, h->theta_host.data(), h->P * sizeof(float), hipMemcpyHostToDevice, stream));
  std::vector<MemberDev> md(h->cfg.K);
  std::vector<int64_t> boff((size_t)h->cfg.L * h->cfg.K);
  for (int k = 0; k < h->cfg.K; ++k) {
    const Member& m = h->mem[k];
    md[k] = MemberDev{m.width, m.dp, m.t, (float)m.scale, (float)m.lr, (float)m.wd, m.act_off,
                      m.toff[2 * m.depth], m.toff[2 * m.depth + 1], m.toff[2 * m.depth - 1],
                      (int64_t)(m.depth - 1) * h->A + m.act_off, (int64_t)(m.depth & 1) * h->A + m.act_off,
                      m.depth, m.d_emb, m.eoff[0], m.eoff[1], m.eoff[2], m.eoff[3], m.h0_off, m.etab_off, m.p_in, 0};
    for (int l = 1; l <= m.depth; ++l) boff[(size_t)(l - 1) * h->cfg.K + k] = m.toff[2 * (l - 1) + 1];
  }
  HIP_TRY(hipMemcpyAsync(h->b.d_mem, md.data(), md.size() * sizeof(MemberDev), hipMemcpyHostToDevice, stream));
  HIP_TRY(hipMemcpyAsync(h->b.d_chunks, h->chunk_tab.data(), h->chunk_tab.size() * 4, hipMemcpyHostToDevice, stream));
  HIP_TRY(hipMemcpyAsync(h->b.d_bias_off, boff.data(), boff.size() * 8, hipMemcpyHostToDevice, stream));
  if (h->prec == Prec::BF16) HIP_TRY(launch_to_shadow(h->b.theta, h->b.shadow, h->P, stream));
  const int rc = upload_plan(h, stream);  // synchronizes the stream
  if (rc) return rc;
  h->t = 0;
  h->bound = true;
  return PACK_OK;
}

int pack_set_active(pack_handle* h, const uint8_t* active, hipStream_t stream) {
  if (!h || !active) return fail(PACK_EINVAL, "NULL argument");
  for (int k = 0; k < h->cfg.K; ++k)
    if (active[k] > 1) return fail(PACK_EINVAL, "active[%d] = %d is not 0 or 1", k, (int)active[k]);
  h->active.assign(active, active + h->cfg.K);
  set_active_ids(h);
  split_members(h);
  if (!h->bound) return PACK_OK;
  // a member that comes back needs keep words for the next step, which were
  // produced (during the last step) for the previous set only
  h->keep_ready = 0;
  return upload_plan(h, stream);
}

int pack_train_step(pack_handle* h, const float* X, const void* y, int64_t N, const int32_t* idx,
                    uint64_t step, float* loss_out, hipStream_t stream) {
  if (!h) return fail(PACK_EINVAL, "handle is NULL");
  if (!h->bound) return fail(PACK_ESTATE, "pack_bind() has not been called");
  if (!X || !y || !idx || !loss_out) return fail(PACK_EINVAL, "NULL device pointer");
  if (N < 1) return fail(PACK_EINVAL, "N=%lld must be positive", (long long)N);
  if (step != h->t + 1) return fail(PACK_ESTATE, "step %llu given, %llu expected", (unsigned long long)step,
                                    (unsigned long long)(h->t + 1));
  if (h->active_ids.empty()) return fail(PACK_ESTATE, "no member is active");
  if (h->stream_rows && (X != h->data_X || N != h->data_N))
    return fail(PACK_EINVAL, "X / N differ from the data bound with pack_bind_data (bind it again, or unbind "
                             "it with X = NULL)");
  const pack_config& c = h->cfg;
  const int nact = (int)h->active_ids.size();
  GemmArgs a = base_args(h);
  a.rows_valid = c.B;
  a.step = as_u32(step);
  const double act_bytes = (double)c.B * h->elt() * [&] {
    double s = 0;
    for (int k : h->active_ids) s += h->mem[k].width;
    return s;
  }();
  auto gemm = [&](OpKind ak, OpKind bk, EpiKind e, const Launch& ln, int layer, hipStream_t s) {
    GemmArgs al = for_launch(a, ln);
    al.layer = layer;
    if (ak == OP_EMB || bk == OP_EMB) set_emb(h, al, X, N, idx, 0);
    return timed(h, gemm_name(h->prec, ak, bk, e), 0, ln.flops, ln.bytes, s,
                 [&] { return launch_gemm(h->prec, ak, bk, e, al, s); });
  };
  // member groups: group 0 on the caller's stream, group g on gstream[g]
  hipStream_t hs[kGroups] = {stream};
  for (int g = 1; g < kGroups; ++g) hs[g] = h->gstream[g];
  const int ng = h->ngroups;
  auto split = [&]() -> hipError_t {
    hipError_t e = hipEventRecord(h->ev_split, stream);
    for (int g = 1; g < ng && e == hipSuccess; ++g) e = hipStreamWaitEvent(hs[g], h->ev_split, 0);
    return e;
  };
  auto merge = [&]() -> hipError_t {
    hipError_t e = hipSuccess;
    for (int g = 1; g < ng && e == hipSuccess; ++g) {
      e = hipEventRecord(h->ev_merge[g], hs[g]);
      if (e == hipSuccess) e = hipStreamWaitEvent(stream, h->ev_merge[g], 0);
    }
    return e;
  };
  int max_dp = 0;
  double nkeep = 0;
  for (int k : h->active_ids) {
    max_dp = std::max(max_dp, h->mem[k].dp);
    nkeep += (double)h->mem[k].depth * h->Bp * h->mem[k].dp / 8;
  }
  // Dropout keep words (Philox, ALU-bound) run on the side stream: normally
  // they were produced during the previous step's backward pass; otherwise
  // (first step, or after a break in the sequence) they are produced now,
  // beside the HBM-bound gather.  Either way the forward GEMMs wait for them.
  const int par = (int)(step & 1);
  auto keep_words = [&](uint64_t s_step, int p) {
    return timed(h, "dropout_words", 1, 0.0, nkeep, h->side, [&] {
      return launch_dropout_words(a.key0, a.key1, as_u32(s_step), h->b.d_mem, nact, c.L, max_dp, h->Bp, c.B,
                                  h->A / 32, h->b.keepw + (size_t)p * c.L * (h->A / 32), h->b.d_active, h->side);
    });
  };
  // indices outside [0, N) are replaced (and flagged) before any kernel reads X or y through them
  HIP_TRY(timed(h, "idx_check", 1, 0.0, 8.0 * c.K * c.B, stream, [&] {
    return launch_idx_check(idx, (int64_t)c.K * c.B, N, h->b.idx_ok, h->b.status, stream);
  }));
  idx = h->b.idx_ok;
  if (h->keep_ready != step) {
    HIP_TRY(hipEventRecord(h->ev_fork, stream));
    HIP_TRY(hipStreamWaitEvent(h->side, h->ev_fork, 0));
    HIP_TRY(keep_words(step, par));
    HIP_TRY(hipEventRecord(h->ev_keep[par], h->side));
  }
  const double bc1 = 1.0 - std::pow(c.beta1, (double)step);
  const double bc2 = 1.0 - std::pow(c.beta2, (double)step);
  const AdamConst ac{(float)c.beta1, (float)c.beta2, (float)c.eps, (float)(1.0 - c.beta1), (float)(1.0 - c.beta2),
                     (float)bc1, (float)std::sqrt(bc2)};
  // Each member group runs its whole chain -- gather, forward GEMMs, head,
  // loss, backward GEMMs with the fused optimizer -- on its own stream; the
  // groups join before the bias/head AdamW.
  HIP_TRY(split());
  for (int hf = 0; hf < ng; ++hf) {
    const hipStream_t s = hs[hf];
    const int gk = h->member0[hf + 1] - h->member0[hf];
    if (h->emb) {
      // the column tables of the group's embeddings from the current parameters;
      // the first-layer forward GEMM produces E from them
      HIP_TRY(emb_tables(h, h->b.d_members + h->member0[hf], h->group[hf], s));
    } else if (!h->stream_rows) {
      // the groups' gathers (HBM-bound) run one after another, so a group's
      // forward GEMMs overlap the next group's gather instead of every group
      // waiting for all the groups' gathers at once
      if (hf > 0) HIP_TRY(hipStreamWaitEvent(s, h->ev_gather[hf - 1], 0));
      HIP_TRY(timed(h, "gather", 1, 0.0, (double)gk * c.B * c.d_in * (4.0 + h->elt()), s, [&] {
        return launch_gather(h->prec, X, c.d_in, h->Pin, idx, c.B, 0, c.B, gk, h->Bp, h->b.H0,
                             h->b.d_members + h->member0[hf], s);
      }));
      HIP_TRY(hipEventRecord(h->ev_gather[hf], s));
    }
    HIP_TRY(hipStreamWaitEvent(s, h->ev_keep[par], 0));
  }
  // The group's gradient sums (hidden biases from the dX partials, head
  // weights and last hidden bias from the head partials, loss and head bias
  // from the per-row values) run as one launch on the side stream once the
  // group's last producer (its last dX launch, or the head backward for
  // one-block packs) is done: off the group's chain; the final bias and head
  // AdamW waits for them.
  auto grad_sums = [&](int hf) -> hipError_t {
    hipError_t e = hipEventRecord(h->ev_bias[hf], hs[hf]);
    if (e == hipSuccess) e = hipStreamWaitEvent(h->side, h->ev_bias[hf], 0);
    if (e != hipSuccess) return e;
    const int t0 = h->sumtile0[hf], t1 = h->sumtile0[hf + 1];
    const double nb = 4.0 * (h->Bp / kPartRows) * 64.0 * (t1 - t0);
    return timed(h, "grad_sums", 1, 0.0, nb, h->side, [&] {
      return launch_grad_sums(h->b.colpart, h->A / kPartRows, h->b.headpart, h->head_rb, h->b.rowloss, h->b.dY,
                              h->b.d_mem, h->b.d_coltiles + t0, t1 - t0, h->Bp, c.B, c.d_out, h->b.d_bias_off, c.K,
                              h->b.grad, loss_out, h->side);
    });
  };
  for (int l = 1; l <= c.L; ++l)
    for (int hf = 0; hf < ng; ++hf)
      HIP_TRY(gemm(l == 1 && h->emb ? OP_EMB : OP_KMAJ, OP_KMAJ, EPI_FWD, h->fwd[par][hf][l - 1], l, hs[hf]));
  for (int hf = 0; hf < ng; ++hf) {
    const hipStream_t s = hs[hf];
    const int32_t* gm = h->b.d_members + h->member0[hf];
    const int gk = h->member0[hf + 1] - h->member0[hf];
    HIP_TRY(timed(h, "head_fwd", 1, 0.0, act_bytes / ng, s, [&] {
      return launch_head_fwd(h->prec, h->task, kHeadTrain, h->b.H, h->b.theta, h->b.d_mem, gk, h->Bp, c.d_out, y,
                             idx, c.B, c.B, 0, 0, h->b.dY, h->b.rowloss, nullptr, gm, s);
    }));
    HIP_TRY(timed(h, "head_bwd", 1, 0.0, 2.0 * act_bytes / ng, s, [&] {
      return launch_head_bwd(h->prec, h->b.H, h->b.theta, h->b.d_mem, h->b.d_headtiles + h->headtile0[hf],
                             h->headtile0[hf + 1] - h->headtile0[hf], h->Bp, h->head_rb, c.d_out, h->b.dY,
                             h->b.dz, h->b.headpart, s);
    }));
    if (c.L == 1) HIP_TRY(grad_sums(hf));
  }
  // the next step's keep words go to the other buffer (last read by the
  // previous step's forward pass) while this step's backward runs
  HIP_TRY(hipEventRecord(h->ev_fork, stream));
  HIP_TRY(hipStreamWaitEvent(h->side, h->ev_fork, 0));
  HIP_TRY(keep_words(step + 1, par ^ 1));
  HIP_TRY(hipEventRecord(h->ev_keep[par ^ 1], h->side));
  h->keep_ready = step + 1;
  for (int l = c.L; l >= 1; --l)
    for (int hf = 0; hf < ng; ++hf) {
      const hipStream_t s = hs[hf];
      // dX_l reads W_l, so it runs before the weight-gradient GEMM updates W_l in place
      if (l > 1) {
        HIP_TRY(gemm(OP_KMAJ, OP_RMAJ, EPI_DX, h->dx[hf][l - 1], l, s));
        if (l == 2) HIP_TRY(grad_sums(hf));
      }
      if (l == 1 && h->emb) {
        // dE = dZ_1 W_1, before W_1 is updated, reduced in the GEMM's epilogue
        // into per-64-row-block gradient sums; then the sums over the blocks
        GemmArgs ae = for_launch(a, h->de[hf]);
        ae.tile_set = TILES_SMALL;
        ae.emb_x = X;
        ae.emb_idx = idx;
        ae.emb_mem = h->b.d_mem;
        ae.emb_d_in = c.d_in;
        ae.emb_tab = h->b.etab;
        HIP_TRY(timed(h, gemm_name(h->prec, OP_KMAJ, OP_RMAJ, EPI_DE), 0, h->de[hf].flops, h->de[hf].bytes, s,
                      [&] { return launch_gemm(h->prec, OP_KMAJ, OP_RMAJ, EPI_DE, ae, s); }));
        const int gk = h->member0[hf + 1] - h->member0[hf];
        double gbytes = 0.0;
        for (int k : h->group[hf]) gbytes += 4.0 * c.d_in * h->mem[k].d_emb * (4.0 * (h->Bp / 64) + 4.0);
        HIP_TRY(timed(h, "embed_grad", 1, 0.0, gbytes, s, [&] {
          return launch_embed_grad(c.d_in, h->Bp, h->b.d_mem, h->b.d_members + h->member0[hf], gk,
                                   max_pin(h, h->group[hf]), h->b.dE, h->b.grad, s);
        }));
      }
      GemmArgs al = for_launch(a, h->dw[hf][l - 1]);
      al.layer = l;
      const OpKind bk = l == 1 && h->emb ? OP_EMB : OP_RMAJ;  // the embedded E is produced in the GEMM
      if (h->muon) {  // the gradient is stored; the Muon step below updates W_l
        HIP_TRY(gemm(OP_RMAJ, bk, EPI_DW, h->dw[hf][l - 1], l, s));
        continue;
      }
      if (bk == OP_EMB) set_emb(h, al, X, N, idx, 0);
      al.theta = h->b.theta;
      al.am = h->b.m;
      al.av = h->b.v;
      al.shadow = h->b.shadow;
      al.adam = ac;
      al.keep_grad = c.keep_grads ? 1 : 0;
      // AdamW fused: the weight update traffic dominates, so the HBM roofline applies
      HIP_TRY(timed(h, gemm_name(h->prec, OP_RMAJ, bk, EPI_DW), 1, h->dw[hf][l - 1].flops, h->dw[hf][l - 1].bytes, s,
                    [&] { return launch_gemm(h->prec, OP_RMAJ, bk, EPI_DW, al, s); }));
    }
  if (h->muon)
    for (int hf = 0; hf < ng; ++hf) HIP_TRY(muon_step(h, a, hf, hs[hf]));
  HIP_TRY(merge());
  // the next step's keep words join the caller's stream too, so that a sync of
  // that stream (or later work on it, such as a re-plan that rewrites the
  // member table the keep-word kernel reads) orders after them
  HIP_TRY(hipEventRecord(h->ev_join, h->side));
  HIP_TRY(hipStreamWaitEvent(stream, h->ev_join, 0));
  double naux = 0;
  for (int k : h->active_ids) {
    const Member& m = h->mem[k];
    naux += (double)m.depth * m.width + (double)c.d_out * m.width + c.d_out;
  }
  HIP_TRY(timed(h, "adamw", 1, 0.0, naux * (h->prec == Prec::BF16 ? 30.0 : 28.0), stream, [&] {
    // biases and head weights: read in fp32 only, so no bf16 copy is written
    return launch_adamw(h->prec, h->b.theta, h->b.grad, h->b.m, h->b.v, nullptr, h->b.d_chunks, h->b.d_aux,
                        h->b.d_mem, h->n_aux_active, ac, stream);
  }));
  h->t = step;
  return PACK_OK;
}

}  // extern "C"

namespace {
// Forward pass without dropout of every active member over rows r0 ..
// r0 + a.rows_valid - 1 of X (N rows): the first layer (on the rows gathered
// once for all members, or, with embeddings, producing each member's
// embedded rows in the GEMM from the column tables, which the caller has
// built), then the hidden layers; the last hidden activations are left in H
// for the head.
hipError_t eval_forward(pack_handle* h, GemmArgs a, const float* X, int64_t N, int64_t r0, hipStream_t stream) {
  const pack_config& c = h->cfg;
  hipError_t e = hipSuccess;
  if (!h->emb)
    e = launch_gather(h->prec, X, c.d_in, h->Pin, nullptr, c.B, r0, a.rows_valid, 1, h->Bp, h->b.H0, nullptr,
                      stream);
  if (e != hipSuccess) return e;
  for (int l = 1; l <= c.L; ++l) {
    for (int hf = 0; hf < (l == 1 ? 1 : h->ngroups); ++hf) {
      GemmArgs al = for_launch(a, l == 1 ? h->fwd1_eval : h->fwd[0][hf][l - 1]);
      al.layer = l;
      const OpKind ak = l == 1 && h->emb ? OP_EMB : OP_KMAJ;
      if (ak == OP_EMB) set_emb(h, al, X, N, nullptr, r0);
      if ((e = launch_gemm(h->prec, ak, OP_KMAJ, EPI_FWD_EVAL, al, stream)) != hipSuccess) return e;
    }
  }
  return hipSuccess;
}
}  // namespace

extern "C" {

int pack_eval_members(pack_handle* h, const float* Xv, const void* yv, int64_t Nv, float* pred_out,
                      double* score_out, hipStream_t stream) {
  if (!h) return fail(PACK_EINVAL, "handle is NULL");
  if (!h->bound) return fail(PACK_ESTATE, "pack_bind() has not been called");
  if (!Xv || !yv || !pred_out || !score_out) return fail(PACK_EINVAL, "NULL device pointer");
  if (Nv < 1) return fail(PACK_EINVAL, "Nv=%lld must be positive", (long long)Nv);
  if (h->active_ids.empty()) return fail(PACK_ESTATE, "no member is active");
  const pack_config& c = h->cfg;
  const int nact = (int)h->active_ids.size();
  GemmArgs a = base_args(h);
  if (h->emb) HIP_TRY(emb_tables(h, h->b.d_active, h->active_ids, stream));
  for (int64_t r0 = 0; r0 < Nv; r0 += h->Bp) {
    a.rows_valid = (int)std::min<int64_t>(h->Bp, Nv - r0);
    HIP_TRY(eval_forward(h, a, Xv, Nv, r0, stream));
    HIP_TRY(launch_head_fwd(h->prec, h->task, kHeadEval, h->b.H, h->b.theta, h->b.d_mem, nact, h->Bp, c.d_out,
                            yv, nullptr, c.B, a.rows_valid, r0, Nv, nullptr, nullptr, pred_out, h->b.d_active,
                            stream));
  }
  HIP_TRY(launch_eval_score(h->task, pred_out, yv, nact, Nv, score_out, h->b.d_active, stream));
  return PACK_OK;
}

int pack_predict(pack_handle* h, const float* X, int64_t N, int32_t mode, float* out, hipStream_t stream) {
  if (!h) return fail(PACK_EINVAL, "handle is NULL");
  if (!h->bound) return fail(PACK_ESTATE, "pack_bind() has not been called");
  if (!X || !out) return fail(PACK_EINVAL, "NULL device pointer");
  if (N < 1) return fail(PACK_EINVAL, "N=%lld must be positive", (long long)N);
  if (mode != PACK_PREDICT_MEMBERS && mode != PACK_PREDICT_ENSEMBLE) return fail(PACK_EINVAL, "unknown mode %d", mode);
  if (h->active_ids.empty()) return fail(PACK_ESTATE, "no member is active");
  const pack_config& c = h->cfg;
  const int nact = (int)h->active_ids.size();
  GemmArgs a = base_args(h);
  if (h->emb) HIP_TRY(emb_tables(h, h->b.d_active, h->active_ids, stream));
  for (int64_t r0 = 0; r0 < N; r0 += h->Bp) {
    a.rows_valid = (int)std::min<int64_t>(h->Bp, N - r0);
    HIP_TRY(eval_forward(h, a, X, N, r0, stream));
    if (mode == PACK_PREDICT_MEMBERS) {
      // member i (i-th active id) writes rows r0.. of out[i, :, :]
      HIP_TRY(launch_head_fwd(h->prec, h->task, kHeadPredict, h->b.H, h->b.theta, h->b.d_mem, nact, h->Bp,
                              c.d_out, nullptr, nullptr, c.B, a.rows_valid, r0, N, nullptr, nullptr, out,
                              h->b.d_active, stream));
    } else {
      // the chunk's member predictions go to the dY buffer ([K, Bp, d_out]), then their mean to out
      HIP_TRY(launch_head_fwd(h->prec, h->task, kHeadPredict, h->b.H, h->b.theta, h->b.d_mem, nact, h->Bp,
                              c.d_out, nullptr, nullptr, c.B, a.rows_valid, 0, h->Bp, nullptr, nullptr, h->b.dY,
                              h->b.d_active, stream));
      HIP_TRY(launch_ensemble_mean(h->b.dY, nact, h->Bp, a.rows_valid, c.d_out, r0, out, stream));
    }
  }
  return PACK_OK;
}

int pack_status(pack_handle* h, uint32_t* flags, hipStream_t stream) {
  if (!h || !flags) return fail(PACK_EINVAL, "NULL argument");
  if (!h->bound) return fail(PACK_ESTATE, "pack_bind() has not been called");
  uint32_t v = 0;
  HIP_TRY(hipMemcpyAsync(&v, h->b.status, sizeof(v), hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipStreamSynchronize(stream));
  if (v) {
    const uint32_t zero = 0;
    HIP_TRY(hipMemcpyAsync(h->b.status, &zero, sizeof(zero), hipMemcpyHostToDevice, stream));
    HIP_TRY(hipStreamSynchronize(stream));
  }
  *flags = v;
  return PACK_OK;
}

static_assert(kMapRows == PACK_BIND_DATA_MAX_B, "the weight-gradient kernels' row table holds a whole batch");

int pack_bind_data(pack_handle* h, const float* X, int64_t N, void* xb, size_t xb_bytes, hipStream_t stream) {
  if (!h) return fail(PACK_EINVAL, "handle is NULL");
  if (!h->bound) return fail(PACK_ESTATE, "pack_bind() has not been called");
  if (!X) {  // unbind: the batch gather feeds the first layer again
    h->stream_rows = false;
    h->data_X = nullptr;
    h->data_N = 0;
    h->xb = nullptr;
    return upload_plan(h, stream);
  }
  if (h->prec != Prec::BF16 || h->emb)
    return fail(PACK_EINVAL, "pack_bind_data needs a bf16 pack without feature embeddings");
  if (N < 1 || !xb) return fail(PACK_EINVAL, "N must be positive and xb set");
  if (h->cfg.B > kMapRows) return fail(PACK_EINVAL, "streamed rows take batches of at most %d rows", kMapRows);
  const size_t need = (size_t)N * h->Pin * 2;
  if (xb_bytes < need) return fail(PACK_EINVAL, "xb has %zu bytes, %zu needed", xb_bytes, need);
  if (reinterpret_cast<uintptr_t>(xb) % 16) return fail(PACK_EINVAL, "xb must be 16-byte aligned");
  if (need + 16 >= ((size_t)1 << 31))
    return fail(PACK_EINVAL, "N x d_in too large for streamed rows (%zu bytes; at most 2 GiB)", need);
  HIP_TRY(launch_rows_to_bf16(X, N, h->cfg.d_in, h->Pin, xb, stream));
  h->stream_rows = true;
  h->data_X = X;
  h->data_N = N;
  h->xb = xb;
  return upload_plan(h, stream);  // the first layer's descriptors read xb through the batch indices
}

int pack_stream_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
  if (!src || !dst) return fail(PACK_EINVAL, "NULL device pointer");
  if (bytes % 16 || reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(dst) % 16)
    return fail(PACK_EINVAL, "bytes and both addresses must be multiples of 16");
  if (bytes == 0) return PACK_OK;
  HIP_TRY(launch_stream_copy(src, dst, (int64_t)(bytes / 16), stream));
  return PACK_OK;
}

int pack_select_workspace_size(int32_t C, int64_t Nv, size_t* bytes) {
  if (!bytes || C < 1 || Nv < 1) return fail(PACK_EINVAL, "C and Nv must be positive");
  const size_t nblk = (size_t)select_blocks(Nv);
  *bytes = (size_t)round_up(Nv * 8, 256) + (size_t)round_up((int64_t)(C * nblk * 8), 256) + 256 + 256;
  return PACK_OK;
}

extern "C++" {
int tabpack::select_with_scratch(pack_handle* h, const float* cand, const void* yv, int32_t C, int64_t Nv,
                                 int32_t m_ens, void* work, size_t work_bytes, int32_t* sel_out, int32_t* n_sel_out,
                                 double* score_out, hipStream_t stream) {
  if (!h) return fail(PACK_EINVAL, "handle is NULL");
  if (!cand || !yv || !work || !n_sel_out || !score_out || (m_ens > 0 && !sel_out))
    return fail(PACK_EINVAL, "NULL device pointer");
  if (C < 1 || C > 65535 || Nv < 1 || m_ens < 0)
    return fail(PACK_EINVAL, "need 1 <= C <= 65535, Nv >= 1 and m_ens >= 0");
  size_t need = 0;
  pack_select_workspace_size(C, Nv, &need);
  if (work_bytes < need) return fail(PACK_EINVAL, "select workspace has %zu bytes, %zu needed", work_bytes, need);
  if (reinterpret_cast<uintptr_t>(work) % 256) return fail(PACK_EINVAL, "select workspace must be 256-byte aligned");
  const int nblk = select_blocks(Nv);
  char* w = static_cast<char*>(work);
  double* sum = reinterpret_cast<double*>(w);
  double* partial = reinterpret_cast<double*>(w + round_up(Nv * 8, 256));
  int32_t* state = reinterpret_cast<int32_t*>(w + round_up(Nv * 8, 256) + round_up((int64_t)C * nblk * 8, 256));
  double* best = reinterpret_cast<double*>(reinterpret_cast<char*>(state) + 256);
  HIP_TRY(launch_select_init(sum, Nv, state, best, n_sel_out, score_out, stream));
  const int iters = std::min(m_ens, C);
  for (int it = 0; it < iters; ++it)
    HIP_TRY(launch_select_iter(h->task, cand, yv, C, Nv, m_ens, sum, partial, nblk, state, best, sel_out, stream));
  HIP_TRY(launch_select_final(state, best, n_sel_out, score_out, stream));
  return PACK_OK;
}
}  // extern "C++"

int pack_select(pack_handle* h, const float* cand, const void* yv, int32_t C, int64_t Nv, int32_t m_ens,
                void* work, size_t work_bytes, int32_t* sel_out, int32_t* n_sel_out, double* score_out,
                hipStream_t stream) {
  return select_with_scratch(h, cand, yv, C, Nv, m_ens, work, work_bytes, sel_out, n_sel_out, score_out, stream);
}

extern "C++" int tabpack::set_error(int code, const char* msg) { return fail(code, "%s", msg); }

int pack_member_param_count(const pack_handle* h, int32_t member, int64_t* count) {
  int rc = check_member(h, member);
  if (rc) return rc;
  if (!count) return fail(PACK_EINVAL, "count is NULL");
  *count = dense_count(h, member);
  return PACK_OK;
}

namespace {
int copy_member(pack_handle* h, int k, const float* dev_base, float* host_out) {
  const int64_t b = member_span_begin(h, k), e = member_span_end(h, k);
  std::vector<float> tmp((size_t)(e - b));
  if (dev_base) {
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(tmp.data(), dev_base + b, tmp.size() * 4, hipMemcpyDeviceToHost));
  } else {
    std::memcpy(tmp.data(), h->theta_host.data() + b, tmp.size() * 4);
  }
  for_each_dense(h, k, [&](int64_t di, int64_t pi) { host_out[di] = tmp[(size_t)(pi - b)]; });
  return PACK_OK;
}
}  // namespace

int pack_get_params(pack_handle* h, int32_t member, float* host_out) {
  int rc = check_member(h, member);
  if (rc) return rc;
  if (!host_out) return fail(PACK_EINVAL, "host_out is NULL");
  return copy_member(h, member, h->bound ? h->b.theta : nullptr, host_out);
}

int pack_set_params(pack_handle* h, int32_t member, const float* host_in) {
  int rc = check_member(h, member);
  if (rc) return rc;
  if (!host_in) return fail(PACK_EINVAL, "host_in is NULL");
  for_each_dense(h, member, [&](int64_t di, int64_t pi) { h->theta_host[(size_t)pi] = host_in[di]; });
  if (h->bound) {
    const int64_t b = member_span_begin(h, member), e = member_span_end(h, member);
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(h->b.theta + b, h->theta_host.data() + b, (size_t)(e - b) * 4, hipMemcpyHostToDevice));
    if (h->prec == Prec::BF16) HIP_TRY(launch_to_shadow(h->b.theta + b, h->b.shadow + b, e - b, 0));
    HIP_TRY(hipDeviceSynchronize());
  }
  return PACK_OK;
}

int pack_get_grads(pack_handle* h, int32_t member, float* host_out) {
  int rc = check_member(h, member);
  if (rc) return rc;
  if (!h->bound) return fail(PACK_ESTATE, "pack_bind() has not been called");
  if (!host_out) return fail(PACK_EINVAL, "host_out is NULL");
  if (!h->cfg.keep_grads) return fail(PACK_ESTATE, "gradients are kept only with pack_config.keep_grads = 1");
  return copy_member(h, member, h->b.grad, host_out);
}

int pack_get_moments(pack_handle* h, int32_t member, float* m_out, float* v_out) {
  int rc = check_member(h, member);
  if (rc) return rc;
  if (!h->bound) return fail(PACK_ESTATE, "pack_bind() has not been called");
  if (!m_out || !v_out) return fail(PACK_EINVAL, "NULL output");
  rc = copy_member(h, member, h->b.m, m_out);
  if (rc) return rc;
  return copy_member(h, member, h->b.v, v_out);
}

int pack_debug_dropout_mask(pack_handle* h, uint64_t step, int32_t layer, int32_t member, uint8_t* dev_out,
                            hipStream_t stream) {
  int rc = check_member(h, member);
  if (rc) return rc;
  if (layer < 1 || layer > h->mem[member].depth)
    return fail(PACK_EINVAL, "layer %d out of [1, %d] for member %d", layer, h->mem[member].depth, member);
  if (!dev_out) return fail(PACK_EINVAL, "dev_out is NULL");
  const Key kd = stream_key(h->cfg.seed, kTagDropout);
  HIP_TRY(launch_dropout_mask(kd.k0, kd.k1, as_u32(step), layer, member, h->mem[member].t, h->cfg.B,
                              h->mem[member].width, dev_out, stream));
  return PACK_OK;
}

int pack_debug_activation(pack_handle* h, int32_t layer, int32_t member, float* host_out) {
  int rc = check_member(h, member);
  if (rc) return rc;
  if (!h->bound) return fail(PACK_ESTATE, "pack_bind() has not been called");
  if (layer < 1 || layer > h->mem[member].depth)
    return fail(PACK_EINVAL, "layer %d out of [1, %d] for member %d", layer, h->mem[member].depth, member);
  if (!host_out) return fail(PACK_EINVAL, "host_out is NULL");
  const Member& m = h->mem[member];
  const size_t n = (size_t)h->Bp * m.dp;
  std::vector<uint8_t> tmp(n * h->elt());
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(tmp.data(), (char*)h->Hl(layer) + (size_t)m.act_off * h->elt(), tmp.size(), hipMemcpyDeviceToHost));
  for (int r = 0; r < h->cfg.B; ++r)
    for (int c = 0; c < m.width; ++c) {
      const size_t i = (size_t)r * m.dp + c;
      float val;
      if (h->prec == Prec::BF16) {
        uint16_t b16;
        std::memcpy(&b16, tmp.data() + 2 * i, 2);
        const uint32_t bits = (uint32_t)b16 << 16;
        std::memcpy(&val, &bits, 4);
      } else {
        std::memcpy(&val, tmp.data() + 4 * i, 4);
      }
      host_out[(size_t)r * m.width + c] = val;
    }
  return PACK_OK;
}

int pack_profile_enable(pack_handle* h, int32_t enable) {
  if (!h) return fail(PACK_EINVAL, "handle is NULL");
  HIP_TRY(hipDeviceSynchronize());
  h->prof = enable != 0;
  h->timed.clear();
  h->pool_used = 0;
  h->groups.clear();
  return PACK_OK;
}

int pack_profile_read(pack_handle* h, pack_kernel_stat* out, int32_t max, int32_t* n) {
  if (!h || !n || (max > 0 && !out)) return fail(PACK_EINVAL, "NULL argument");
  std::vector<ProfGroup> g = h->groups;
  for (ProfGroup& x : g) x.launches = 0, x.total_ms = 0.0;
  // launch intervals on a common time base (the first recorded event), to
  // measure each kernel's busy time: the union of its launches' intervals,
  // which differs from the summed durations when launches of concurrent
  // member groups overlap
  std::vector<std::vector<std::pair<double, double>>> iv(g.size());
  for (const TimedLaunch& t : h->timed) {
    HIP_TRY(hipEventSynchronize(t.stop));
    float ms = 0.0f, t0 = 0.0f, t1 = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, t.start, t.stop));
    HIP_TRY(hipEventElapsedTime(&t0, h->timed.front().start, t.start));
    HIP_TRY(hipEventElapsedTime(&t1, h->timed.front().start, t.stop));
    g[t.group].launches += 1;
    g[t.group].total_ms += ms;
    iv[t.group].push_back({t0, t1});
  }
  *n = (int32_t)g.size();
  for (int i = 0; i < (int)g.size() && i < max; ++i) {
    pack_kernel_stat& s = out[i];
    std::memset(&s, 0, sizeof s);
    snprintf(s.name, sizeof s.name, "%s", g[i].name.c_str());
    s.kind = g[i].kind;
    s.launches = g[i].launches;
    s.total_ms = g[i].total_ms;
    s.flops = g[i].launches ? g[i].flops / g[i].launches : 0.0;
    s.bytes = g[i].launches ? g[i].bytes / g[i].launches : 0.0;
    std::sort(iv[i].begin(), iv[i].end());
    double busy = 0.0, a = 0.0, b = -1.0;
    for (const auto& x : iv[i]) {
      if (x.first > b) {
        if (b > a) busy += b - a;
        a = x.first;
        b = x.second;
      } else {
        b = std::max(b, x.second);
      }
    }
    if (b > a) busy += b - a;
    s.busy_ms = busy;
  }
  return PACK_OK;
}

}  // extern "C"
