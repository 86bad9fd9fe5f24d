// Device views of the trie, the per-user decoding state and the drafted tree.
#pragma once
#include <hip/hip_runtime.h>
#include "common.h"

namespace atspeed {

constexpr int kMaxPar = 128;  // parents per level (>= max(K, N))
constexpr int kMaxSel = 128;  // selected per level (>= max(K, N))

// Item trie: node 0 is the root; the children of node n are the nodes
// first[n] .. first[n] + cnt[n] - 1, sorted by code.
struct TrieDev {
  const int* code;
  const int* first;
  const int* cnt;
};

// Per-user state: current item level t and the target beams Y_t.
struct StateDev {
  int* t;           // [B]
  int* nb;          // [B] beams held
  uint32_t* path;   // [B, K] path keys
  int* trie;        // [B, K] trie node of each beam
  float* score;     // [B, K] target cumulative log-prob
  float* qscore;    // [B, K] draft cumulative log-prob (drafting)
  int* beam_slot;   // [B, K] tree slot of each beam's last node (t > 0)
  int* steps;       // [B] speculative steps run
  int* npath;       // [B] tree nodes holding the Y_t paths
  int* nfwd;        // [B] tree nodes forwarded by verify (depth < L)
  int K, gamma;
};

struct TreeDev {
  int max_nodes;
  int* n_nodes;
  int* token;
  int* parent;
  int* depth;
  float* q_score;
  uint32_t* tpath;  // derived: path key of each node
  int* ttrie;       // derived: trie node of each node
};

// Per-user candidate scratch of the relaxed modes (max_cand entries per user).
struct CandBuf {
  uint32_t* path;
  int* par;
  int* cidx;
  float* sp;
  float* sq;
  __host__ __device__ CandBuf offset(size_t o) const { return CandBuf{path + o, par + o, cidx + o, sp + o, sq + o}; }
};

// Relaxed-mode parameters and buffers.
struct RelaxArgs {
  int mode;                 // 1 EXACT, 2 PAPER
  float tau;
  uint32_t k0, k1;          // Philox key
  int N;
  float* zq;                // [B, L+1] draft log-normaliser of each drafted level
  int* slot_node;           // [B, L+1, K] EXACT: tree slot of every drafted slot
  unsigned long long* keys; // [B, max_cand]
};

void launch_draft_relaxed(const StateDev& s, const TreeDev& tr, const TrieDev& trie, const float* lpq,
                          const float* rootq, int nitem, int item_base, int codebook, int L, int j, int* lvl_lo,
                          int* lvl_hi, const CandBuf& cb, int max_cand, const RelaxArgs& ra, int B, hipStream_t st);
void launch_verify_relaxed(const StateDev& s, const TreeDev& tr, const TrieDev& trie, const float* lpt,
                           const float* roott, const float* lpq, const float* rootq, int nitem, int codebook, int L,
                           const CandBuf& cb, int max_cand, const RelaxArgs& ra, int* accepted, int* t_after, int B,
                           hipStream_t st);

void launch_tree_from_beams(const StateDev& s, const TreeDev& tr, const TrieDev& trie, int B, int item_base,
                            int codebook, int L, hipStream_t st);
// Appends the current beams Y_t of every user to a [B][K*L][L] sequence buffer
// (codes, lengths t) at the user's count n[u] and advances it.
void launch_append_beams(const StateDev& s, int B, int L, int* items, int* lens, int* n, hipStream_t st);
void launch_tree_index(const TreeDev& tr, const TrieDev& trie, const StateDev& s, int B, int item_base, int codebook,
                       int L, int* err, hipStream_t st);
// Row plan of one forward: nodes with slot in [lo[u], hi[u]) of every user, users
// in order (with idx: entries [lo[u], hi[u]) of the user's node list idx[u*max_nodes..]);
// writes rows.M and (if maxrows) the largest per-user row count.
void launch_plan_tree(const TreeDev& tr, const int* lo, const int* hi, int B, int P, const Rows& rows, int* maxrows,
                      hipStream_t st, const int* idx = nullptr);
// Tree-KV reuse across the verifies of one decode: matches the nodes to forward
// (s.nfwd) against the previous tree's forwarded nodes by (depth, path key),
// writing src (previous slot or -1), the list idx of nodes still to forward and
// its length cnt (prev_n null: nothing matches); then copies the matched nodes'
// per-layer K/V rows and log-prob rows between the two buffer sets.
void launch_carry_match(const TreeDev& tr, const StateDev& s, const uint32_t* prev_tpath, const int* prev_depth,
                        const int* prev_n, int* src, int* idx, int* cnt, int B, hipStream_t st);
void launch_carry_copy(const int* src, const int* nfwd, int B, int Tm, int n_layers, size_t layer_bytes,
                       int row_bytes, const void* k_old, const void* v_old, void* k_new, void* v_new,
                       const float* lp_old, float* lp_new, int nitem, hipStream_t st);
// Prefill rows sharing the first S positions: the longest prefix all users have
// in common is computed on the device (launch_common_prefix); user 0 forwards all
// P positions, the others P - S, and their first S K/V rows are user 0's
// (launch_broadcast_prefix_kv, once per layer after the K/V projection).
void launch_common_prefix(const int* prefix, int B, int P, int* out, hipStream_t st);
void launch_plan_prefix(const int* prefix, int B, int P, int S, const Rows& rows, hipStream_t st);
// Outputs of a decode from the state: items [B, K, L], scores [B, K], n_items [B] (device).
void launch_write_lists(const StateDev& s, int B, int K, int L, int32_t* items, float* scores, int32_t* n_items,
                        hipStream_t st);
void launch_broadcast_prefix_kv(void* pk, void* pv, int B, int H, size_t head_bytes, size_t shared_bytes,
                                hipStream_t st);
void launch_draft_beam_scores(const StateDev& s, const TreeDev& tr, const float* lpq, const float* rootq, int nitem,
                              int codebook, int L, int B, hipStream_t st);
void launch_draft_select(const StateDev& s, const TreeDev& tr, const TrieDev& trie, const float* lpq,
                         const float* rootq, int nitem, int item_base, int codebook, int L, int j, int N, int* lvl_lo,
                         int* lvl_hi, unsigned long long* keys, int max_cand, int B, hipStream_t st);
void launch_verify_strict(const StateDev& s, const TreeDev& tr, const TrieDev& trie, const float* lpt,
                          const float* roott, int nitem, int codebook, int L, unsigned long long* keys, int max_cand,
                          int* accepted, int* t_after, int B, hipStream_t st);

}  // namespace atspeed
