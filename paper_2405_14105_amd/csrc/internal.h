// Internal declarations shared by the kernel translation units and the
// runtime.  gfx950 (CDNA4) only: 64-wide wavefronts, bf16/fp32 MFMA.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dsi {

// ----------------------------------------------------------------- layouts
//
// Streaming tile ("packed") layout of a GEMM weight W [N, K] (rows = output
// features): tiles of 16 rows x 32 k, stored [Nb][Kb][64 lanes][8 elems] so
// that one wavefront loads one tile as 64 x 16 B (bf16) contiguous bytes --
// exactly the A-operand fragment of a 16x16x32 MFMA: lane l holds row
// (l % 16) and k = 8 * (l / 16) + e, e = 0..7.  Rows and k beyond N, K are 0.
//
// Activation pack for a GEMM input X [M, K]: [Mt][Kb][64][8] with lane l
// holding token (l % 16) and the same k mapping -- the B-operand fragment.
// For bf16 weights an fp32 activation x is carried as two bf16 packs,
// hi = bf16(x) and lo = bf16(x - hi), and each tile costs two MFMAs, so the
// GEMM is accurate to ~2^-17 relative instead of bf16's 2^-9.  For fp32
// weights the pack holds fp32 and the fp32 MFMA 16x16x4 is used.
//
// MFMA output (16x16, fp32): lane l holds rows 4*(l/16) + j, j = 0..3, of
// column l % 16 -- four output features of one token.
//
// Row order inside a 16-row tile for two fused epilogues:
//  * RoPE pairing (Q and K sections of the fused QKV weight): tile row
//    4g + jj holds pair index 2g + (jj & 1) and half (jj >> 1), so a lane
//    owns both members (x_j, x_{j+hd/2}) of two rotary pairs.
//  * SwiGLU interleave (fused gate/up weight): tile row 4g + jj holds FFN
//    feature 8*nb + 2g + (jj & 1), gate for jj < 2 and up for jj >= 2.
//
// KV cache of one layer and window: K [n_kv][max_len_pad][hd] and the value
// cache transposed in blocks of 32 positions, V^T [n_kv][max_len_pad/32][hd][32]
// (max_len_pad is a multiple of 64).  Both attention MFMAs read 16
// contiguous bytes per lane, and the keys and values of one 32-key step are
// two contiguous blocks (32 x hd elements each), which keeps long-prefix
// attention on long DRAM bursts.

enum WType : int { W_F32 = 0, W_BF16 = 1 };

constexpr int kTileRows = 16;
constexpr int kTileK = 32;
constexpr int kMaxMt = 4;          // at most 64 rows per forward chunk
constexpr int kMaxRows = kMaxMt * 16;

// gemm epilogues
// EPI_PART stores split s of a K-split GEMM into its own partial buffer
// (out + s * part_stride); the residual stream is updated by the next
// RMSNorm, which folds x += sum_s partial_s in split order.
// EPI_RESID (no K split) adds the product to the residual stream in place,
// x[m][n] += y, writes the next RMSNorm's input before scaling, x * gain,
// into the consumer's activation pack, and stores the sum of x^2 over the
// 16 features of each n-block in ssq[m * Nb + nb].  The consuming
// GEMM (GemmArgs::ssq) forms the RMSNorm scale of each row from those sums
// and applies it to its accumulators: W (x * g) / rms(x) = W RMSNorm(x).
// EPI_PARTRES: EPI_PART, then the last of the S split workgroups of each
// n-block group to finish (an arrival counter per group, reset by that
// workgroup) folds x += sum_s partial_s in split order for the group's
// features and writes what EPI_RESID writes (x, x * gain into the pack,
// ssq), plus an optional copy of x.
enum Epi : int { EPI_STORE = 0, EPI_PART = 1, EPI_QKV = 2, EPI_SILU = 3, EPI_RESID = 4, EPI_PARTRES = 5 };

struct PackRef {        // an activation pack (hi/lo bf16, or fp32 in hi)
  void* hi;
  void* lo;
  int Kb;               // k-blocks of the consuming GEMM
};

struct RowMap {         // token row m -> (window, row within window, position)
  const int* lens;      // device window lengths
  int window0;
  int rows_per_window;  // R
  // nullable: token-tree rows, RoPE position lens[w] + depth[m] (the node's
  // depth in its tree) instead of lens[w] + (m % R).  The cache slot of row
  // m is lens[w] + (m % R) either way.
  const int* depth;
};

// KV cache of one (layer, window, KV head): a region of maxlen * hd elements
// in blocks of 32 positions.  K is stored per block as [hd/32][32 positions]
// [32 dims] and V transposed per block as [hd][32 positions], so the K (and
// V) fragments of one 32-key attention step are whole 128-byte lines of one
// contiguous 32 * hd block.  Element offsets of (position p, dim d):
__host__ __device__ inline size_t kc_off(int p, int d, int hd) {
  return ((size_t)(p >> 5) * hd + (d & ~31)) * 32 + (size_t)(p & 31) * 32 + (d & 31);
}
__host__ __device__ inline size_t vc_off(int p, int d, int hd) {
  return ((size_t)(p >> 5) * hd + d) * 32 + (p & 31);
}

struct EpiArgs {
  int kind;
  // EPI_STORE: out [M][ld]; EPI_PART: out [S][part_stride] holding [M][ld]
  float* out;
  int ld;
  size_t part_stride;
  int n_valid;          // logical N (features) -- outputs beyond are dropped
  // EPI_QKV
  float* q_out;         // [M][n_heads*hd]
  void* kcache;         // layer base: [windows][n_kv] regions of maxlen*hd (kc_off)
  void* vcache;         // layer base: [windows][n_kv] regions of maxlen*hd (vc_off)
  int kv_bf16;
  int n_heads, n_kv, hd, maxlen;
  const float2* rope;   // [M][hd/2] (cos, sin)
  RowMap rows;
  // EPI_SILU (pack, ff), EPI_RESID (pack, x, gain, ssq; out unused)
  PackRef pack;
  int ff;
  float* x;             // [M][ld] residual stream, updated in place
  const float* gain;    // [ld] gain of the RMSNorm that consumes x
  float* ssq;           // [M][Nb] per-n-block sums of x^2
  int* cnt;             // EPI_PARTRES: [n-block groups] arrival counters (zero between launches)
  float* copy;          // EPI_PARTRES: nullable [M][ld] copy of the folded x
};

struct GemmArgs {
  const void* W;
  // Nullable: the same weights in the ring (stream) layout of the role's
  // RingCfg; one-row-tile launches that set it run the ring kernel.
  const void* Ws = nullptr;
  int ring_nk = 0;      // k-blocks per wave of that layout
  int ring_nbw = 0;     // n-blocks per workgroup of that layout
  const void* Xhi;
  const void* Xlo;
  int Nb, Kb, M;
  int S;                // K splits across workgroups (EPI_PART only; else 1)
  int G = 1;            // n-block group of the packed layout (wtile_index)
  EpiArgs epi;
  // optional RMSNorm of the input rows (the pack holds x * gain): the
  // accumulators of row m are scaled by 1/sqrt(sum_nb ssq[m][nb] / norm_d + eps)
  const float* ssq;     // [M][ssq_n] or nullptr
  int ssq_n, norm_d;
  float eps;
};
// K split the launcher uses for an EPI_PART GEMM of this shape
int gemm_part_splits(int wtype, int Nb, int Kb, int mt);
// Packed weight layout.  A matrix of Nb n-blocks x Kb k-blocks is stored as
// 1 KB tiles (16 rows x 32 k); n-blocks are grouped G at a time and the
// tiles of a group are k-block major, [group][kb][n-block in group] (the
// last group may hold fewer than G), so the G tiles of one k-block of a
// group are contiguous.  G = 1 is the plain [nb][kb] order.
__host__ __device__ inline size_t wtile_index(int nb, int kb, int Nb, int Kb, int G) {
  const int g = nb / G, j = nb - g * G;
  const int gs = Nb - g * G < G ? Nb - g * G : G;
  return (size_t)g * G * Kb + (size_t)kb * gs + j;
}
// Group size the GEMM of this role and shape reads best: the n-blocks per
// workgroup of its one-row-tile launch (bf16 gate/up and LM head), else 1.
int gemm_wgroup(int wtype, int epi_kind, int Nb);
constexpr int kMaxSplits = 4;

// Ring layout of a GEMM weight for one-row-tile launches (gemm.hip,
// k_gemm_ring).  A launch has `wgs` workgroups of kRingWaves waves; workgroup
// g*S + s owns n-blocks [g*nbw, g*nbw + nbw) and the K split s, i.e. k-blocks
// [s*kRingWaves*nk, (s+1)*kRingWaves*nk), of which wave w takes the nk
// consecutive ones starting at s*kRingWaves*nk + w*nk.  Every wave's tiles
// are one contiguous run in the order it consumes them, k-block major:
//   tile (wave, i, j) = ((wg * kRingWaves + w) * nk + i) * nbw + j
// (1 KB each); tiles past the matrix (n-block >= Nb or k-block >= Kb) are 0.
constexpr int kRingWaves = 8;
struct RingCfg {
  int nbw = 0;          // n-blocks per workgroup (0: no ring layout for this role)
  int nk = 0;           // k-blocks per wave
  int S = 1;            // K splits across workgroups
  int wgs = 0;          // workgroups of a launch
  __host__ __device__ size_t tiles() const { return (size_t)wgs * kRingWaves * nk * nbw; }
};
// Ring layout of a role's weight (epi_kind) of Nb x Kb tiles split S ways
// along K; false when the role has none (the launch uses the packed layout).
bool ring_config(int wtype, int epi_kind, int Nb, int Kb, int S, RingCfg* out);
// src: the packed layout (wtile_index with group G) -> dst: ring layout
hipError_t launch_restream(const void* src, int Nb, int Kb, int G, const RingCfg& c, void* dst,
                           hipStream_t s);

// launchers (gemm.hip)
hipError_t launch_gemm(int wtype, int mt, const GemmArgs& a, hipStream_t s);

// prepack (elementwise.hip): src [N][K] row-major (device), dst packed
// (wtile_index with dst_Nb n-blocks in groups of G).  rowmap: 0 plain, 1
// rope-paired (QKV sections), 2 gate/up interleave (which = 0 gate, 1 up).
// dst_nb0: first destination n-block.
hipError_t launch_prepack(int wtype, const void* src, int N, int K, void* dst, int Kb,
                          int dst_nb0, int rowmap, int hd, int which, int dst_Nb, int G,
                          hipStream_t s);

// embed gather + RMSNorm + pack + rope table (elementwise.hip)
struct EmbedArgs {
  const int* tokens;    // [M]
  const void* E;        // [V][d] wdtype
  int wtype;
  int V, d, M;
  float* x;             // [M][d] residual out
  const float* gain;    // first layer attention-norm gain
  float eps;
  PackRef pack;
  float2* rope;         // [M][hd/2]
  int hd;
  double log2_base;
  RowMap rows;
  int* err;
  float* hidden0;       // optional copy of x (diagnostics)
};
hipError_t launch_embed_norm(const EmbedArgs& a, hipStream_t s);

// Residual fold and RMSNorm of x rows into a pack: x += sum of the S partial
// buffers delta + s * delta_stride (S may be 0), then pack rmsnorm(x) * gain;
// also an optional diagnostic copy of the updated x.
hipError_t launch_rmsnorm_pack(float* x, const float* delta, int S, size_t delta_stride, int M, int d,
                               const float* gain, float eps, int wtype, PackRef pack, float* copy_out,
                               hipStream_t s);

// attention (attention.hip)
struct AttnArgs {
  const float* q;       // [M][n_heads*hd]
  const void* kc;       // layer base
  const void* vc;
  RowMap rows;
  int n_windows;
  int n_heads, n_kv, maxlen;
  int n_qtiles, chunk, n_chunks;
  float scale;
  float* part_o;        // [windows*n_kv][qtiles][chunks][16][hd]
  float2* part_ml;      // [windows*n_kv][qtiles][chunks][16]
  PackRef out;          // O-projection input pack
  int wtype;
  // nullable: token-tree rows.  Row m may attend to window key L + j
  // (j < R) only if bit j of anc[m] is set (its ancestors and itself); the
  // cached prefix [0, L) is visible to every row.
  const unsigned long long* anc;
  int waves;            // waves per workgroup: kAttnWaves, or 4; chunk % (32 waves) == 0
};
constexpr int kAttnWaves = 8;                       // waves per attention workgroup (default)
hipError_t launch_attention(int kv_bf16, int hd, const AttnArgs& a, hipStream_t s);

// verification (verify.hip)
struct VerifyArgs {
  int B, k, V;
  const float* logits;  // [B*(k+1)][V]
  const int* tokens;    // [B][k+1]
  const float* q;       // [B][k][V]
  const float* u;       // [B][k+1]
  double temperature;
  int greedy;
  int commit;
  int* lens;            // nullable: window lengths (commit)
  int window0;
  int* n_out;
  int* tok_out;
  int* err;
  // workspace
  double2* part;        // [B*(k+1)][C]: (max, sumexp)
  float2* part_arg;     // [B*(k+1)][C]: (max value, index as float bits)
  double2* rowstat;     // [B*(k+1)]: (M, S)
  int* rowarg;          // [B*(k+1)]
  int4* decision;       // [B]: (n, row, residual, err)
  double2* csum;        // [B][C]: (sum r, sum p)
  int C;                // chunks per row
};
constexpr int kVerifyChunk = 4096;  // vocabulary entries per chunk (256 thr x 16)

// drafter sampling (draft.hip): q = softmax(z / T) stored fp32 and one draft
// drawn from it by inverse CDF
struct DraftArgs {
  const float* logits;  // [V] drafter logits of the row that ends the context
  int V, C;
  double temperature;
  const float* u;       // [1] the uniform of this draft
  float* q_out;         // [V] the stored distribution
  int* tok_out;         // [1] the draft
  double2* part;        // workspace [C]: chunk (max z/T, sum exp)
  double* csum;         // workspace [C]: chunk sums of the stored q
};
size_t draft_workspace_bytes(int V);
hipError_t launch_draft_sample(DraftArgs a, void* ws, hipStream_t s);
size_t verify_workspace_bytes(int rows, int B, int V);
void verify_bind_workspace(VerifyArgs& a, void* ws, int rows, int B, int V);
hipError_t launch_verify(const VerifyArgs& a, hipStream_t s);
// the per-(row, chunk) statistics pass of launch_verify alone (B*(k+1) rows)
hipError_t launch_verify_rowstats(const VerifyArgs& a, hipStream_t s);

// token trees (tree.hip).  B windows of R nodes; node 0 of each tree is the
// window's w0, node i > 0 has parent[i] in [0, i).
struct TreeArgs {
  int B, R, V, C;
  const int* tokens;            // [B][R]
  const int* parent;            // [B][R]
  int* depth;                   // [B*R]  (prep output)
  unsigned long long* anc;      // [B*R]  (prep output)
  int* bad;                     // [B]    (prep output: invalid parent array)
  const float2* part_arg;       // [B*R][C] chunk (max, argmax) of the logits
  int* path;                    // [B][R] accepted node path, -1 beyond n
  int* n_out;
  int* tok_out;
  int commit;
  int* lens;
  int window0;
  int* err;
  int4* decision;               // [B]: (n, L before commit, bad, 0)
};
hipError_t launch_tree_prep(const TreeArgs& a, hipStream_t s);
hipError_t launch_tree_decide(const TreeArgs& a, hipStream_t s);
// move the K/V rows of each window's accepted path to consecutive slots
// L+1..L+n (after launch_tree_decide).  kc / vc: cache bases, layer stride
// layer_elems, window stride win_elems (elements).
hipError_t launch_tree_compact(const TreeArgs& a, int kv_bf16, void* kc, void* vc, int n_layers,
                               size_t layer_elems, size_t win_elems, int n_kv, int hd, int maxlen,
                               hipStream_t s);

// KV and misc (elementwise.hip)
hipError_t launch_kv_rollback(int* lens, int window, int new_len, int* err, hipStream_t s);
hipError_t launch_kv_set(int* lens, int window, int new_len, hipStream_t s);
hipError_t launch_kv_add_checked(int* lens, int window, const int* tokens, int n, int V, int* err,
                                 hipStream_t s);
hipError_t launch_kv_copy(int to_cache, int kv_bf16, void* kc, void* vc, int n_kv, int hd,
                          int maxlen, int len, void* dk, void* dv, hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
// streaming read of kStreamWorkgroups x 8 waves, each over per_wave_vec
// 16-byte vectors of buf (diagnostics: dsi_profile_stream)
constexpr int kStreamWorkgroups = 256;      // default grid
constexpr int kStreamMaxWorkgroups = 4096;
hipError_t launch_stream_read(const void* buf, size_t per_wave_vec, int workgroups, int nontemporal, void* sink,
                              hipStream_t s);
// NaN into rows [lens[window], maxlen) of every layer's K and V of one window
// (kc / vc: the window's layer-0 base; layers layer_stride elements apart)
hipError_t launch_kv_poison(int kv_bf16, void* kc, void* vc, size_t layer_stride, int n_layers, int n_kv, int hd,
                            int maxlen, const int* lens, int window, hipStream_t s);
hipError_t launch_copy_rows(const float* src, float* dst, size_t n, hipStream_t s);

}  // namespace dsi
