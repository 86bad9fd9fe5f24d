// Host-side launchers of the device kernels (one translation unit per family).
#pragma once
#include <hip/hip_runtime.h>
#include "common.h"
#include "select.h"

namespace atspeed {

enum GemmKind { GEMM_STORE = 0, GEMM_RESID = 1, GEMM_GU = 2, GEMM_QKV = 3 };

struct GemmCall {
  int kind;
  bool bf16;
  const void* A; int lda;
  int Mmax; const int* Mdev;
  int N, K;
  const void* w0; const void* w1; const void* w2;
  int split;                 // QKV: d_model; GU: d_ffn
  float* out; int ldo;       // STORE / RESID
  float* part;               // bf16 RESID: k split at K/2; the second half's product [Mmax, ldo] fp32 goes here
  void* hout;                // GU output [M, f]
  void* q; void* kdst; void* vdst;
  const float* cosT; const float* sinT;   // fp32 path: [max_pos, d_head/2] each
  const float* ropeT;        // bf16 path: [max_pos][16][4] (cos, sin) of rotary index 16*b + i at [pos][i][b] (0 past d_head/2)
  Rows rows;
  int kv_mode, Pmax, d, dh, H;
  float* scratch;            // fp32 path: [Mmax, N] product
};
hipError_t gemm(const GemmCall& g, hipStream_t st);

// Attention of every row over its visible prefix-cache keys and tree keys.
struct AttnCall {
  bool bf16;
  const void* q;        // [M, d]
  const void* pk; const void* pv;   // prefix cache of this layer [B][H][Pmax][dh]
  const void* tk; const void* tv;   // tree KV of this layer [slot][d] (may be null)
  void* out;            // [M, d]
  Rows rows;
  int Mmax, B, Tq;      // Tq: max rows per user (grid bound)
  int H, dh, d, Pmax;
};
hipError_t attention(const AttnCall& a, hipStream_t st);

// Misc
hipError_t gather_kv_rows(const void* kc, const void* vc, const Rows& rows, int rmax, int kv_mode, int H, int dh,
                          int Pmax, void* ko, void* vo, hipStream_t st);
hipError_t embed(bool bf16, const void* emb, const Rows& rows, int Mmax, int d, float* x, hipStream_t st);
// add (may be null): a k-split GEMM's second partial product, added to x first;
// the sum is written back to x when row_index is null.
hipError_t rmsnorm(bool bf16, float* x, const float* add, const int* Mdev, int Mmax, int d, const float* g, void* out,
                   const int* row_index, hipStream_t st);
hipError_t log_softmax_rows(const float* logits, const int* Mdev, int Mmax, int n, const int* dst_index,
                            float* lp, float* logits_copy, hipStream_t st);

// Draft alignment (AtSpeed-S / AtSpeed-R training of the draft's item head).
struct AlignRows {
  const int* Mdev;           // [1] context rows of the draft forward
  const int* user;           // [Mmax] user of each row
  const int* slot;           // [Mmax] tree slot (u * max_nodes + s) of each row
  const float* lq;           // draft log-probs by slot [B * max_nodes, nitem]
  const float* lq_root;      // [B, nitem]
  const float* lp;           // target log-probs by slot
  const float* lp_root;
  const float* ctx_weight;   // [B * max_nodes] weight of each node as a context
  const float* label_weight; // [B * max_nodes] weight of each node as its parent's label
  const float* root_weight;  // [B]
  const float* log_pK;       // [B, L]
};
void launch_align_tree(const int* items, const int* lens, const int* n_items, int S, const TreeDev& tr,
                       const TrieDev& trie, int B, int L, int item_base, int codebook, float* ctx_weight,
                       float* label_weight, float* root_weight, int* kslot, int* err, hipStream_t st);
void launch_align_logpk(const int* items, const int* n_items, const int* kslot, const float* lp, const float* root,
                        int B, int S, int L, int codebook, int nitem, float* log_pK, hipStream_t st);
void launch_align_grad(const AlignRows& ar, const TrieDev& trie, const TreeDev& tr, int B, int M, int nitem,
                       int codebook, int L, int K, int mode, float alpha, float* dz, float* loss_rows,
                       hipStream_t st);
// log((1 - lam) exp(lq) + lam exp(lp)) into lq, rows [0, nrows[u]) of each user (all if null).
void launch_mix_logprobs(float* lq, const float* lp, const int* nrows, int B, int rows_per_user, int nitem, float lam,
                         hipStream_t st);
void launch_head_grad(bool bf16, const float* dz, const void* h_root, const void* h_rows, const int* Mdev, int B,
                      int nitem, int d, float* dW, hipStream_t st);
void launch_align_hidden(bool bf16, const void* h_root, const void* h_rows, const int* slot, const int* Mdev, int B,
                         int M, int d, float* out, hipStream_t st);
void launch_adamw(bool bf16, float* master, float* m, float* v, const float* g, void* head, size_t n, float lr,
                  float b1, float b2, float eps, float wd, int step, hipStream_t st);

}  // namespace atspeed
