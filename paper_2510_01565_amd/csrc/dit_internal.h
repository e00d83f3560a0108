// Internal structures shared by the host orchestration and the HIP kernels.
// Everything a kernel needs about a packed batch travels by value in its
// arguments (BatchMeta), so no metadata is ever uploaded to the device.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dit.h"

namespace dit {

constexpr int kMaxReq = DIT_MAX_REQUESTS;

// Row bookkeeping of a packed batch.
//  stream-major rows: [text of req 0 .. text of req n-1 | image of req 0 .. image of req n-1]
//  joint positions:   [req 0: text, image | req 1: text, image | ...]  (the order of dit_attention)
//  padded positions:  [req 0: image, text, pad | req 1: image, text, pad | ...]  (Q / K / V^T of the step)
struct BatchMeta {
  int n_req;
  int T_txt;                 // total text rows
  int T_img;                 // total image rows
  int T;                     // T_txt + T_img
  int txt_off[kMaxReq + 1];  // text row offsets (stream-major)
  int img_off[kMaxReq + 1];  // image row offsets, relative to T_txt
  int joint_off[kMaxReq + 1];
  int pad_off[kMaxReq + 1];  // joint offsets with every request padded to a multiple of 64
  int n_txt[kMaxReq];
  int grid_w[kMaxReq];
};

constexpr int kSeqPad = 64;

struct RowInfo {
  int req;     // request index
  int is_img;  // 1 for image tokens
  int local;   // index inside the request's text or image rows
};

__host__ __device__ inline RowInfo row_info(const BatchMeta& m, int R) {
  RowInfo ri;
  if (R < m.T_txt) {
    int r = 0;
    while (r + 1 < m.n_req && R >= m.txt_off[r + 1]) ++r;
    ri.req = r;
    ri.is_img = 0;
    ri.local = R - m.txt_off[r];
  } else {
    int Ri = R - m.T_txt;
    int r = 0;
    while (r + 1 < m.n_req && Ri >= m.img_off[r + 1]) ++r;
    ri.req = r;
    ri.is_img = 1;
    ri.local = Ri - m.img_off[r];
  }
  return ri;
}

// Position of a row inside the padded layout of Q, K and V^T that the step
// uses: request r occupies [pad_off[r], pad_off[r + 1]) with its image tokens
// first, then its text tokens.  Attention does not depend on the order of the
// tokens inside a request; image-first starts both parts on a 16-token group
// whenever the image count is a multiple of 16 (the (res/16)^2 grid of every
// resolution that is a multiple of 64), so the QKV epilogue writes V^T in
// whole 16-token groups whatever the text length.
__host__ __device__ inline int req_images(const BatchMeta& m, int r) { return m.img_off[r + 1] - m.img_off[r]; }

__host__ __device__ inline int padded_pos(const BatchMeta& m, const RowInfo& ri) {
  return m.pad_off[ri.req] + (ri.is_img ? 0 : req_images(m, ri.req)) + ri.local;
}

// stream-major row of position q (0 <= q < L_r) of request r in that layout
__host__ __device__ inline int padded_to_row(const BatchMeta& m, int r, int q) {
  const int ni = req_images(m, r);
  return q < ni ? m.T_txt + m.img_off[r] + q : m.txt_off[r] + (q - ni);
}

// Column of padded position `pos` in V^T.  Inside every aligned group of 16
// keys the middle two quads are swapped (keys 4-7 <-> 8-11), the order in
// which one 32x32 score fragment holds them; an involution.
__host__ __device__ inline int vt_slot(int pos) { return (pos & ~12) | ((pos & 4) << 1) | ((pos & 8) >> 1); }


// ----------------------------------------------------------------------------
// GEMM epilogues: Y = A W^T + bias, then one of
enum EpiMode : int {
  EPI_STORE_F32 = 0,  // out[m, n] = y (fp32)
  EPI_STORE_T = 1,    // out[m, n] = y (storage type: bf16 or fp32)
  EPI_GELU = 2,       // out[m, col0 + n] = GELU(y)
  EPI_RESID = 3,      // out[m, n] (fp32) += gate[req(m), n] * y
  EPI_QKV = 4         // n < n_qkv: Q/K/V scatter with 2-D RoPE on image rows;
                      // n >= n_qkv: gelu_out[m, gelu_col0 + n - n_qkv] = GELU(y)
};

struct EpiArgs {
  int mode;
  int row_base;         // stream-major row of the group's row 0 (request lookup)
  const void* bias;     // [N], weight type, may be null
  void* out;            // already offset to the group's row 0
  long ldo;
  int col0;
  const float* mods;    // EPI_RESID: gate = mods[req * mods_ld + gate_off + n]
  int mods_ld;
  int gate_off;
  // EPI_QKV
  void* q;              // [heads][T][d]
  void* k;              // [heads][T][d]
  void* vt;             // [heads][d][T], column vt_slot(padded position)
  int T;                // padded joint length (pad_off[n_req]): Q / K rows per head
  long vt_ld;           // row pitch of V^T in elements (>= T)
  int hidden;
  int head_dim;
  int n_qkv;            // 3 * hidden
  const float2* rope;   // [DIT_MAX_GRID][head_dim / 4] (cos, sin)
  void* gelu_out;
  long gelu_ld;
  int gelu_col0;
};

struct GemmGroup {
  const void* A;  // [M, K], lda
  long lda;
  const void* W;  // [N, K], ldw
  long ldw;
  int M;
  int K;
  EpiArgs epi;
};

// Split of K across blocks for launches with too few output tiles: every
// tile's K range is cut into sk_p equal pieces run by sk_p blocks; each piece
// publishes its fp32 partial sums, and the last piece of a tile to arrive adds
// all of them in piece order and runs the epilogue.
constexpr int kSplitMaxTiles = 1024;                   // arrival counters in the workspace
constexpr long kSplitPartBytes = 96L * 1024 * 1024;    // partial-sum slots in the workspace

struct GemmProblem {
  int N;
  int n_groups;  // 1 or 2
  GemmGroup g[2];
  BatchMeta meta;
  float* sk_part;  // kSplitPartBytes of workspace, or null: never split
  int* sk_cnt;     // kSplitMaxTiles arrival counters, zero before and after every launch
  int sk_p;        // pieces per tile, set by the launcher (1: no split)
};

// ----------------------------------------------------------------------------
// launchers (return hipError_t of the launch)
hipError_t launch_gemm_bf16(const GemmProblem& p, hipStream_t s);
hipError_t launch_gemm_f32(const GemmProblem& p, hipStream_t s);
// name of the kernel configuration launch_gemm_bf16 picks for p
const char* gemm_bf16_config_name(const GemmProblem& p);
// whether the launch model predicts p's two groups to finish sooner as two
// launches of one group each (the caller then launches them in turn)
bool gemm_bf16_split_groups(const GemmProblem& p);

// Attention over the requests of a batch.  Token p of request r
// (0 <= p < L_r, in the order of o_stream_major) is read from Q/K row qk_off[r] + p and from V^T
// column vt_off[r] + p; V^T columns of a request are padded to a multiple of
// 64 (vt_off from pad_off) so that a 64-key tile never leaves the buffer.
struct AttnArgs {
  const void* q;
  long q_tok, q_head;   // element strides
  const void* k;
  long k_tok, k_head;
  const void* vt;       // Vt[h][dd][vt column]
  long vt_head, vt_d;
  void* o;
  long o_tok, o_head;
  int o_stream_major;   // 1: token p is padded position p of the step's layout, output row padded_to_row(r, p);
                        // 0: token p is joint position p, output row joint_off[r] + p
  int heads;
  int head_dim;
  float scale;          // 1/sqrt(head_dim)
  int qk_off[kMaxReq + 1];
  int vt_off[kMaxReq + 1];
  BatchMeta meta;
  // Scratch for splitting the key range of a launch's last, partly filled
  // round of query tiles (bf16, head dim 128): at least
  // attn_split_bytes(meta, heads, head_dim) bytes, or null (never split; the
  // output bits then do not depend on how many other tiles share the launch).
  float* split_buf;
  // set by the launcher: this launch covers query-tile units
  // [unit0, unit0 + units); kv_pieces > 1 splits each unit's keys into that
  // many ranges whose unnormalised partial results go to split_buf
  int unit0, units, kv_pieces;
};
hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t s);
// bytes of split_buf the bf16 launcher may use for this batch (0: it never splits)
size_t attn_split_bytes(const BatchMeta& m, int heads, int head_dim);
hipError_t launch_attention_f32(const AttnArgs& a, hipStream_t s);

// elementwise / reduction kernels
hipError_t launch_rope_table(float2* table, int head_dim, float theta, hipStream_t s);
hipError_t launch_timestep_embed(float* e, int n_req, const float* t_host, int dim, hipStream_t s);
// y[r, o] = sum_k W[o, k] * act(x[r, k]) + b[o]; act 0 = identity, 1 = SiLU
hipError_t launch_gemv(int wdtype, const void* W, const void* b, const float* x, long ldx, int n_req,
                       int K, int N, int act, float* y, long ldy, hipStream_t s);
// adaLN LayerNorm of rows [row_begin, row_end) of X (fp32, ld H) into out (row 0 = row_begin)
hipError_t launch_ln_modulate(int out_dtype, const float* X, int H, int row_begin, int row_end,
                              const BatchMeta& meta, const float* mods, int mods_ld, int shift_txt,
                              int scale_txt, int shift_img, int scale_img, float eps, void* out,
                              long ldo, hipStream_t s);
hipError_t launch_euler(int dtype, void* x, const void* v, int channels, const BatchMeta& meta,
                        const float* dt_host, hipStream_t s);
// v [T_joint, heads, d] (joint order) -> vt [heads][d][pad_off[n]] at columns vt_slot(padded position)
hipError_t launch_v_transpose(int dtype, const void* v, const BatchMeta& meta, int heads, int d, void* vt,
                              hipStream_t s);
// n ints at p set to zero (a fill kernel, so a captured graph holds no memset node)
hipError_t launch_zero_i32(int* p, int n, hipStream_t s);
// zeroes the V^T columns of the padding keys of every request (padded positions >= the request length)
hipError_t launch_vt_pad_zero(int dtype, void* vt, long ld, const BatchMeta& meta, int heads, int d, hipStream_t s);

}  // namespace dit
