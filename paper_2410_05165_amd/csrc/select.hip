// Tree bookkeeping, trie-constrained beam selection and strict acceptance.
//
// A sequence of codes is packed into a 32-bit path key, code of item level l in
// byte 3-l, so comparing path keys of equal depth compares the sequences
// lexicographically.  A candidate's 64-bit selection key is
//   (~orderkey(score) << 32) | pathkey
// whose ascending order is: higher score first, then lexicographically smaller
// sequence (the pinned tie-break).  Keys are unique because paths are.
// TopK is a radix select on those keys (8 bits per pass, 256-bin LDS histogram)
// followed by a rank sort of the K survivors, one workgroup per user.
#include "common.h"
#include "select.h"
#include "select_dev.h"

namespace atspeed {

// ---------------------------------------------------------------- tree kernels

// Paths of the current beams Y_t (depths 1..t), deduplicated and level-ordered,
// become the first nodes of each user's tree; beam_slot[k] is beam k's node.
// The nodes are looked up while the tree is built, so their depth, path key
// and trie node are mirrored in LDS (a lookup then costs no round trip to
// memory): at most K <= 128 beams times t < L <= 4 levels of nodes.
constexpr int kMaxPathNodes = kMaxSel * 3;
__global__ void tree_from_beams_kernel(StateDev s, TreeDev tr, TrieDev trie, int item_base, int codebook, int L) {
  __shared__ int dep_s[kMaxPathNodes], trie_s[kMaxPathNodes];
  __shared__ uint32_t path_s[kMaxPathNodes];
  const int u = blockIdx.x;
  if (threadIdx.x != 0) return;
  const int t = s.t[u];
  const int nb = s.nb[u];
  int n = 0;
  const size_t tb = (size_t)u * tr.max_nodes;
  const int K = s.K;
  if (t > 0 && t < L) {
    for (int l = 1; l <= t; ++l) {
      const uint32_t mask = l == 4 ? 0xFFFFFFFFu : ~(0xFFFFFFFFu >> (8 * l));
      for (int k = 0; k < nb; ++k) {
        const uint32_t pre = s.path[u * K + k] & mask;
        int found = -1;
        for (int i = 0; i < n; ++i)
          if (dep_s[i] == l && path_s[i] == pre) { found = i; break; }
        if (found < 0) {
          int parent = -1, ptrie = 0;
          if (l > 1) {
            const uint32_t pm = ~(0xFFFFFFFFu >> (8 * (l - 1)));
            for (int i = 0; i < n; ++i)
              if (dep_s[i] == l - 1 && path_s[i] == (pre & pm)) { parent = i; break; }
            ptrie = parent >= 0 ? trie_s[parent] : 0;  // found: the prefix was added at level l - 1
          }
          const int code = path_code(pre, l - 1);
          const int node = trie_child(trie, ptrie, code);
          tr.token[tb + n] = item_base + codebook * (l - 1) + code;
          tr.parent[tb + n] = parent;
          tr.depth[tb + n] = l;
          tr.q_score[tb + n] = 0.f;
          tr.tpath[tb + n] = pre;
          tr.ttrie[tb + n] = node;
          dep_s[n] = l;
          path_s[n] = pre;
          trie_s[n] = node;
          found = n++;
        }
        if (l == t) s.beam_slot[u * K + k] = found;
      }
    }
  }
  tr.n_nodes[u] = n;
  s.npath[u] = n;
}

// Derived per-node data of a caller or draft tree: path key, trie node, ancestors;
// validation; number of nodes to forward (depth < L, a prefix of the level order).
__global__ void tree_index_kernel(TreeDev tr, TrieDev trie, StateDev s, int item_base, int codebook, int L, int* err) {
  const int u = blockIdx.x;
  const size_t tb = (size_t)u * tr.max_nodes;
  const int n = s.t[u] >= L ? 0 : tr.n_nodes[u];
  __shared__ int nfwd, bad;
  if (threadIdx.x == 0) {
    nfwd = n;
    bad = 0;
  }
  __syncthreads();
  if (n < 0 || n > tr.max_nodes) {
    if (threadIdx.x == 0) {
      atomicOr(err, 1);
      s.nfwd[u] = 0;   // nothing of this user is forwarded
    }
    return;
  }
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    int chain[4], dep = tr.depth[tb + i], cur = i, ok = dep >= 1 && dep <= L;
    for (int l = dep; ok && l >= 1; --l) {
      if (cur < 0 || cur > i || tr.depth[tb + cur] != l) { ok = 0; break; }
      chain[l - 1] = cur;
      const int p = tr.parent[tb + cur];
      if (l == 1 ? p != -1 : (p < 0 || p >= cur)) { ok = 0; break; }
      cur = p;
    }
    if (ok && i > 0 && tr.depth[tb + i - 1] > dep) ok = 0;  // level order
    uint32_t path = 0;
    int node = 0;
    for (int l = 1; ok && l <= dep; ++l) {
      const int code = tr.token[tb + chain[l - 1]] - item_base - codebook * (l - 1);
      if (code < 0 || code >= codebook) { ok = 0; break; }
      node = trie_child(trie, node, code);
      if (node < 0) { ok = 0; break; }
      path = path_with(path, l - 1, code);
    }
    if (!ok) {
      atomicOr(err, 1);
      bad = 1;
      continue;
    }
    tr.tpath[tb + i] = path;
    tr.ttrie[tb + i] = node;
    if (dep == L) atomicMin(&nfwd, i);
  }
  __syncthreads();
  // A user whose tree has any malformed node forwards nothing: the row planner
  // walks parents, depths and tokens of the forwarded nodes, and only
  // validated ones keep those walks inside the tree and the tables.
  if (threadIdx.x == 0) s.nfwd[u] = bad ? 0 : nfwd;
}

// Beam slots of Y_t in a caller tree (verify): every beam path must be a node of depth t.
__global__ void find_beam_slots_kernel(TreeDev tr, StateDev s, int L, int* err) {
  const int u = blockIdx.x;
  const int t = s.t[u];
  if (t <= 0 || t >= L) return;
  const size_t tb = (size_t)u * tr.max_nodes;
  const int n = tr.n_nodes[u];
  if (n < 0 || n > tr.max_nodes) return;   // flagged by tree_index_kernel
  for (int k = threadIdx.x; k < s.nb[u]; k += blockDim.x) {
    const uint32_t p = s.path[u * s.K + k];
    int found = -1;
    for (int i = 0; i < n; ++i)
      if (tr.depth[tb + i] == t && tr.tpath[tb + i] == p) { found = i; break; }
    if (found < 0) atomicOr(err, 2);
    s.beam_slot[u * s.K + k] = found;
  }
}

// Rows of one forward: nodes with slot in [lo[u], hi[u]) of every user, users in
// order; with idx, entries [lo[u], hi[u]) of the user's node list idx instead.
__global__ void plan_tree_rows_kernel(TreeDev tr, const int* lo, const int* hi, const int* idx, int B, int P,
                                      Rows rows, int* maxrows) {
  __shared__ int off[1025];
  if (threadIdx.x == 0) {
    int acc = 0, mx = 0;
    for (int u = 0; u < B; ++u) {
      off[u] = acc;
      rows.user_off[u] = acc;
      const int n = max(0, hi[u] - lo[u]);
      acc += n;
      mx = max(mx, n);
    }
    off[B] = acc;
    rows.user_off[B] = acc;
    *rows.M = acc;
    if (maxrows) *maxrows = mx;
  }
  __syncthreads();
  // every row in parallel: its user is the last u with off[u] <= r (users
  // without rows share their offset with the next one and are never picked)
  const int total = off[B];
  for (int r = threadIdx.x; r < total; r += blockDim.x) {
    int ul = 0, uh = B - 1;
    while (ul < uh) {
      const int mid = (ul + uh + 1) >> 1;
      if (off[mid] <= r) ul = mid; else uh = mid - 1;
    }
    const int u = ul;
    const size_t tb = (size_t)u * tr.max_nodes;
    {
      const int e = lo[u] + (r - off[u]);
      const int s = idx ? idx[tb + e] : e;
      const int dep = tr.depth[tb + s];
      rows.user[r] = u;
      rows.token[r] = tr.token[tb + s];
      rows.pos[r] = P + dep - 1;
      rows.slot[r] = (int)(tb + s);
      rows.nctx[r] = P;
      int cur = s;
      for (int l = dep; l >= 1; --l) {
        rows.anc[r * 4 + l - 1] = (int)(tb + cur);
        cur = tr.parent[tb + cur];
      }
      for (int l = dep; l < 4; ++l) rows.anc[r * 4 + l] = 0;
      rows.nanc[r] = dep;
    }
  }
}

// Tree nodes whose target K/V the previous verify of the same decode already
// holds.  A node's K/V and log-probs depend only on the prefix and the node's
// path (its position is P + depth - 1), so a node of this tree with the same
// (depth, path) as a node forwarded (or carried) by the previous verify takes
// that node's values instead of a forward.  For every node i < nfwd[u]:
// src[i] = its slot in the previous tree or -1; idx lists, in order, the nodes
// with src -1 (the rows to forward) and cnt[u] counts them.  np_prev null: no
// previous tree, everything is forwarded.
__global__ void __launch_bounds__(256) carry_match_kernel(TreeDev tr, StateDev s, const uint32_t* prev_tpath,
                                                          const int* prev_depth, const int* prev_n, int* src,
                                                          int* idx, int* cnt) {
  const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t tb = (size_t)u * tr.max_nodes;
  const int n = s.nfwd[u];
  const int np = prev_n ? prev_n[u] : 0;
  __shared__ int wsum[4];
  int base = 0;
  for (int c0 = 0; c0 < n; c0 += 256) {   // uniform trip count over the block
    const int i = c0 + tid;
    int j = -1;
    if (i < n) {
      const int dep = tr.depth[tb + i];
      const uint32_t key = tr.tpath[tb + i];
      for (int q = 0; q < np; ++q)
        if (prev_depth[tb + q] == dep && prev_tpath[tb + q] == key) { j = q; break; }
      src[tb + i] = j;
    }
    // order-preserving compaction of the nodes to forward
    const bool fwd = i < n && j < 0;
    const unsigned long long m = __ballot(fwd);
    const int rank = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wave] = __popcll(m);
    __syncthreads();
    int before = base;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    if (fwd) idx[tb + before + rank] = i;
    base += wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
  }
  if (tid == 0) cnt[u] = base;
}

// Copies the carried nodes' K/V rows (every layer) and log-prob rows from the
// previous verify's buffers into this verify's, at the nodes' new slots.  One
// block per slot; the two buffer sets are disjoint.
__global__ void __launch_bounds__(256) carry_copy_kernel(const int* src, const int* nfwd, int Tm, int n_layers,
                                                         size_t layer_bytes, int row_bytes, const char* k_old,
                                                         const char* v_old, char* k_new, char* v_new,
                                                         const float* lp_old, float* lp_new, int nitem) {
  const int node = blockIdx.x, u = node / Tm, i = node - u * Tm;
  if (i >= nfwd[u]) return;
  const int j = src[node];
  if (j < 0) return;
  const size_t from = (size_t)u * Tm + j;
  const int nv = row_bytes / 16;
  for (int l = 0; l < n_layers; ++l) {
    const size_t o_new = l * layer_bytes + (size_t)node * row_bytes, o_old = l * layer_bytes + from * row_bytes;
    for (int e = threadIdx.x; e < nv; e += blockDim.x) {
      reinterpret_cast<uint4*>(k_new + o_new)[e] = reinterpret_cast<const uint4*>(k_old + o_old)[e];
      reinterpret_cast<uint4*>(v_new + o_new)[e] = reinterpret_cast<const uint4*>(v_old + o_old)[e];
    }
  }
  for (int e = threadIdx.x; e < nitem; e += blockDim.x)
    lp_new[(size_t)node * nitem + e] = lp_old[from * nitem + e];
}

// Length of the prefix every user shares with user 0 (tokens equal at every
// position before it), at most P.
__global__ void common_prefix_kernel(const int* prefix, int B, int P, int* out) {
  __shared__ int len;
  if (threadIdx.x == 0) len = P;
  __syncthreads();
  const int total = (B - 1) * P;
  for (int i = threadIdx.x; i < total; i += blockDim.x) {
    const int u = 1 + i / P, p = i % P;
    if (prefix[u * P + p] != prefix[p]) atomicMin(&len, p);
  }
  __syncthreads();
  if (threadIdx.x == 0) *out = len;
}

// Rows of the prefill: user 0 forwards positions 0..P-1, every other user only
// S..P-1 (its first S positions are user 0's, whose K/V it copies).
__global__ void plan_prefix_rows_kernel(const int* prefix, int B, int P, int S, Rows rows) {
  const int own = P - S;
  const int total = P + (B - 1) * own;
  for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < total; r += gridDim.x * blockDim.x) {
    int u, p;
    if (r < P) {
      u = 0;
      p = r;
    } else {
      const int q = r - P;
      u = 1 + q / own;
      p = S + q % own;
    }
    rows.user[r] = u;
    rows.token[r] = prefix[u * P + p];
    rows.pos[r] = p;
    rows.slot[r] = -1;
    rows.nctx[r] = p + 1;
    rows.nanc[r] = 0;
    if (r == 0) {
      for (int v = 0; v < B; ++v) rows.user_off[v] = v == 0 ? 0 : P + (v - 1) * own;
      rows.user_off[B] = total;
      *rows.M = total;
    }
  }
}

// K/V of the first S positions of user 0 to users 1..B-1, one layer of the
// prefix cache [user][head][Pmax][d_head] (16-byte chunks).
__global__ void broadcast_prefix_kv_kernel(unsigned char* pk, unsigned char* pv, int B, int H, size_t head_bytes,
                                           size_t shared_bytes) {
  const size_t chunks = shared_bytes / 16;
  const size_t per_user = (size_t)H * chunks;
  const size_t total = (size_t)(B - 1) * per_user * 2;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const size_t kv = i / ((size_t)(B - 1) * per_user), rest = i % ((size_t)(B - 1) * per_user);
    const size_t u = 1 + rest / per_user, hc = rest % per_user;
    const size_t h = hc / chunks, c = hc % chunks;
    unsigned char* base = kv == 0 ? pk : pv;
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(base + h * head_bytes) + c;
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(base + (u * H + h) * head_bytes) + c;
    *dst = *src;
  }
}

// ---------------------------------------------------------------- draft
// Draft score of every beam of Y_t: sum of draft log-probs along its path.
__global__ void draft_beam_scores_kernel(StateDev s, TreeDev tr, const float* lpq, const float* rootq, int nitem,
                                         int codebook, int L) {
  const int u = blockIdx.x;
  const int t = s.t[u];
  if (t >= L) return;
  for (int k = threadIdx.x; k < s.nb[u]; k += blockDim.x) {
    float acc = 0.f;
    if (t > 0) {
      int chain[4], cur = s.beam_slot[u * s.K + k];
      for (int l = t; l >= 1; --l) { chain[l - 1] = cur; cur = tr.parent[(size_t)u * tr.max_nodes + cur]; }
      const uint32_t p = s.path[u * s.K + k];
      for (int l = 1; l <= t; ++l) {
        const float* row = l == 1 ? rootq + (size_t)u * nitem
                                  : lpq + ((size_t)u * tr.max_nodes + chain[l - 2]) * nitem;
        acc += row[codebook * (l - 1) + path_code(p, l - 1)];
      }
    }
    s.qscore[u * s.K + k] = acc;
  }
}

// One drafted level: TopN over the extensions of the previous level (level 1:
// the beams of Y_t), appended to the tree; lvl[u] = [begin, end) of the new nodes.
__global__ void __launch_bounds__(256)
draft_select_kernel(StateDev s, TreeDev tr, TrieDev trie, const float* lpq, const float* rootq, int nitem,
                    int item_base, int codebook, int L, int j, int N, int* lvl_lo, int* lvl_hi,
                    unsigned long long* keys_all, int max_cand) {
  __shared__ SelShared sh;
  __shared__ uint32_t ppath[kMaxPar];
  __shared__ float pscore[kMaxPar];
  __shared__ int ptrie[kMaxPar], pslot[kMaxPar];
  __shared__ const float* plp[kMaxPar];
  __shared__ unsigned long long sel[2 * kMaxSel];
  const int u = blockIdx.x, tid = threadIdx.x;
  const int t = s.t[u];
  const int J = min(s.gamma, L - t);
  const size_t tb = (size_t)u * tr.max_nodes;
  if (t >= L || j > J) {
    if (tid == 0) { lvl_lo[u] = tr.n_nodes[u]; lvl_hi[u] = tr.n_nodes[u]; }
    return;
  }
  int npar;
  if (j == 1) {
    npar = t == 0 ? 1 : s.nb[u];
    for (int i = tid; i < npar; i += blockDim.x) {
      if (t == 0) { ppath[i] = 0; pscore[i] = 0.f; ptrie[i] = 0; pslot[i] = -1; plp[i] = rootq + (size_t)u * nitem; }
      else {
        const int sl = s.beam_slot[u * s.K + i];
        ppath[i] = s.path[u * s.K + i]; pscore[i] = s.qscore[u * s.K + i]; ptrie[i] = s.trie[u * s.K + i];
        pslot[i] = sl; plp[i] = lpq + (tb + sl) * nitem;
      }
    }
  } else {
    const int a = lvl_lo[u];
    npar = lvl_hi[u] - a;
    for (int i = tid; i < npar; i += blockDim.x) {
      const int sl = a + i;
      ppath[i] = tr.tpath[tb + sl]; pscore[i] = tr.q_score[tb + sl]; ptrie[i] = tr.ttrie[tb + sl];
      pslot[i] = sl; plp[i] = lpq + (tb + sl) * nitem;
    }
  }
  __syncthreads();
  unsigned long long* keys = keys_all + (size_t)u * max_cand;
  const int lvl0 = t + j - 1;
  const int n = gen_candidates(trie, npar, ppath, pscore, ptrie, plp, lvl0, codebook, keys, sh);
  const int ns = select_smallest(keys, n, N, sel, sh);
  const int base = tr.n_nodes[u];
  for (int i = tid; i < ns; i += blockDim.x) {
    const unsigned long long k = sel[i];
    const uint32_t path = (uint32_t)k;
    const int code = path_code(path, lvl0);
    const uint32_t ppre = lvl0 == 0 ? 0u : (path & ~(0xFFFFFFFFu >> (8 * lvl0)));
    int pi = 0;
    for (int q = 0; q < npar; ++q) if (ppath[q] == ppre) { pi = q; break; }
    const int sl = base + i;
    tr.token[tb + sl] = item_base + codebook * lvl0 + code;
    tr.parent[tb + sl] = pslot[pi];
    tr.depth[tb + sl] = lvl0 + 1;
    tr.q_score[tb + sl] = key_score(k);
    tr.tpath[tb + sl] = path;
    tr.ttrie[tb + sl] = trie_child(trie, ptrie[pi], code);
  }
  __syncthreads();
  if (tid == 0) {
    tr.n_nodes[u] = base + ns;
    lvl_lo[u] = base;
    lvl_hi[u] = base + ns;
  }
}

// ---------------------------------------------------------------- strict verify
// Algorithm 1 per user, on target log-probs by tree slot (lpt) and at the root.
__global__ void __launch_bounds__(256)
verify_strict_kernel(StateDev s, TreeDev tr, TrieDev trie, const float* lpt, const float* roott, int nitem,
                     int codebook, int L, unsigned long long* keys_all, int max_cand, int* accepted_out,
                     int* t_after_out) {
  __shared__ SelShared sh;
  __shared__ uint32_t ppath[kMaxPar];
  __shared__ float pscore[kMaxPar];
  __shared__ int ptrie[kMaxPar], pslot[kMaxPar];
  __shared__ const float* plp[kMaxPar];
  __shared__ unsigned long long sel[2 * kMaxSel];
  __shared__ int ok_s;
  constexpr int kTreeLds = 1024;     // nodes whose (depth, path) are staged in LDS
  __shared__ uint32_t tpath_s[kTreeLds];
  __shared__ int depth_s[kTreeLds];
  const int u = blockIdx.x, tid = threadIdx.x;
  const int t = s.t[u];
  const int K = s.K;
  if (t >= L) {
    if (tid == 0) { if (accepted_out) accepted_out[u] = -1; if (t_after_out) t_after_out[u] = t; }
    return;
  }
  const size_t tb = (size_t)u * tr.max_nodes;
  const int J = min(s.gamma, L - t);
  int npar = t == 0 ? 1 : s.nb[u];
  for (int i = tid; i < npar; i += blockDim.x) {
    if (t == 0) { ppath[i] = 0; pscore[i] = 0.f; ptrie[i] = 0; pslot[i] = -1; plp[i] = roott + (size_t)u * nitem; }
    else {
      const int sl = s.beam_slot[u * K + i];
      ppath[i] = s.path[u * K + i]; pscore[i] = s.score[u * K + i]; ptrie[i] = s.trie[u * K + i];
      pslot[i] = sl; plp[i] = lpt + (tb + sl) * nitem;
    }
  }
  // the drafted nodes, read once: each selected path is looked up among them
  // at every level (from global memory that lookup was a chain of dependent loads)
  const int ntree = tr.n_nodes[u];
  const bool staged = ntree <= kTreeLds;
  if (staged)
    for (int i = tid; i < ntree; i += blockDim.x) { tpath_s[i] = tr.tpath[tb + i]; depth_s[i] = tr.depth[tb + i]; }
  __syncthreads();
  unsigned long long* keys = keys_all + (size_t)u * max_cand;
  int accepted = 0, t_after = t;
  for (int j = 1; j <= J + 1; ++j) {
    const int lvl0 = t + j - 1;        // 0-based level of the codes chosen now
    if (lvl0 >= L) break;
    const bool bonus = (j == J + 1);   // every drafted level accepted, item not complete
    const int n = gen_candidates(trie, npar, ppath, pscore, ptrie, plp, lvl0, codebook, keys, sh);
    const int ns = select_smallest(keys, n, K, sel, sh);
    // T_j and its membership in the drafted level t+j
    if (tid == 0) ok_s = 1;
    __syncthreads();
    uint32_t mypath = 0; float myscore = 0.f; int mytrie = -1, myslot = -1;
    if (tid < ns) {
      const unsigned long long k = sel[tid];
      mypath = (uint32_t)k;
      myscore = key_score(k);
      const int code = path_code(mypath, lvl0);
      const uint32_t ppre = lvl0 == 0 ? 0u : (mypath & ~(0xFFFFFFFFu >> (8 * lvl0)));
      int pi = 0;
      for (int q = 0; q < npar; ++q) if (ppath[q] == ppre) { pi = q; break; }
      mytrie = trie_child(trie, ptrie[pi], code);
      if (!bonus) {
        for (int i = 0; i < ntree; ++i) {
          const int di = staged ? depth_s[i] : tr.depth[tb + i];
          const uint32_t pi = staged ? tpath_s[i] : tr.tpath[tb + i];
          if (di == lvl0 + 1 && pi == mypath) { myslot = i; break; }
        }
        if (myslot < 0) atomicAnd(&ok_s, 0);
      }
    }
    __syncthreads();
    const int ok = ok_s;
    if (tid < ns) {
      ppath[tid] = mypath; pscore[tid] = myscore; ptrie[tid] = mytrie; pslot[tid] = myslot;
      plp[tid] = myslot >= 0 ? lpt + (tb + myslot) * nitem : nullptr;
    }
    npar = ns;
    __syncthreads();
    if (bonus) { accepted = J; t_after = lvl0 + 1; break; }
    if (lvl0 + 1 == L) { accepted = ok ? j : j - 1; t_after = L; break; }
    if (!ok) { accepted = j - 1; t_after = lvl0 + 1; break; }
  }
  // new state: T (ppath, pscore, ptrie)
  for (int i = tid; i < npar; i += blockDim.x) {
    s.path[u * K + i] = ppath[i];
    s.score[u * K + i] = pscore[i];
    s.trie[u * K + i] = ptrie[i];
  }
  if (tid == 0) {
    s.nb[u] = npar;
    s.t[u] = t_after;
    s.steps[u] += 1;
    if (accepted_out) accepted_out[u] = accepted;
    if (t_after_out) t_after_out[u] = t_after;
  }
}

// Appends each user's current beams Y_t (codes of depths 1..t, zero past t) to
// items [B][K*L][L] / lens [B][K*L] at the user's count n[u], which it advances
// (one level of a target-only beam search; K*L rows hold every level).
__global__ void append_beams_kernel(StateDev s, int L, int* __restrict__ items, int* __restrict__ lens,
                                    int* __restrict__ n) {
  const int u = blockIdx.x, K = s.K;
  const int t = s.t[u], nb = s.nb[u], base = n[u];
  const size_t rb = (size_t)u * K * L;
  for (int k = threadIdx.x; k < nb; k += blockDim.x) {
    if (base + k >= K * L) break;
    const uint32_t p = s.path[u * K + k];
    for (int l = 0; l < L; ++l) items[(rb + base + k) * L + l] = l < t ? path_code(p, l) : 0;
    lens[rb + base + k] = t;
  }
  __syncthreads();
  if (threadIdx.x == 0) n[u] = min(base + nb, K * L);
}

// ---------------------------------------------------------------- launchers
void launch_tree_from_beams(const StateDev& s, const TreeDev& tr, const TrieDev& trie, int B, int item_base,
                            int codebook, int L, hipStream_t st) {
  hipLaunchKernelGGL(tree_from_beams_kernel, dim3(B), dim3(64), 0, st, s, tr, trie, item_base, codebook, L);
}
void launch_append_beams(const StateDev& s, int B, int L, int* items, int* lens, int* n, hipStream_t st) {
  hipLaunchKernelGGL(append_beams_kernel, dim3(B), dim3(64), 0, st, s, L, items, lens, n);
}
void launch_tree_index(const TreeDev& tr, const TrieDev& trie, const StateDev& s, int B, int item_base, int codebook,
                       int L, int* err, hipStream_t st) {
  hipLaunchKernelGGL(tree_index_kernel, dim3(B), dim3(256), 0, st, tr, trie, s, item_base, codebook, L, err);
  hipLaunchKernelGGL(find_beam_slots_kernel, dim3(B), dim3(64), 0, st, tr, s, L, err);
}
void launch_plan_tree(const TreeDev& tr, const int* lo, const int* hi, int B, int P, const Rows& rows, int* maxrows,
                      hipStream_t st, const int* idx) {
  hipLaunchKernelGGL(plan_tree_rows_kernel, dim3(1), dim3(1024), 0, st, tr, lo, hi, idx, B, P, rows, maxrows);
}
void launch_carry_match(const TreeDev& tr, const StateDev& s, const uint32_t* prev_tpath, const int* prev_depth,
                        const int* prev_n, int* src, int* idx, int* cnt, int B, hipStream_t st) {
  hipLaunchKernelGGL(carry_match_kernel, dim3(B), dim3(256), 0, st, tr, s, prev_tpath, prev_depth, prev_n, src, idx,
                     cnt);
}
void launch_carry_copy(const int* src, const int* nfwd, int B, int Tm, int n_layers, size_t layer_bytes,
                       int row_bytes, const void* k_old, const void* v_old, void* k_new, void* v_new,
                       const float* lp_old, float* lp_new, int nitem, hipStream_t st) {
  hipLaunchKernelGGL(carry_copy_kernel, dim3(B * Tm), dim3(256), 0, st, src, nfwd, Tm, n_layers, layer_bytes,
                     row_bytes, (const char*)k_old, (const char*)v_old, (char*)k_new, (char*)v_new, lp_old, lp_new,
                     nitem);
}
void launch_common_prefix(const int* prefix, int B, int P, int* out, hipStream_t st) {
  hipLaunchKernelGGL(common_prefix_kernel, dim3(1), dim3(1024), 0, st, prefix, B, P, out);
}
void launch_plan_prefix(const int* prefix, int B, int P, int S, const Rows& rows, hipStream_t st) {
  const int total = P + (B - 1) * (P - S);
  int blocks = std::max(1, std::min(1024, (total + 255) / 256));
  hipLaunchKernelGGL(plan_prefix_rows_kernel, dim3(blocks), dim3(256), 0, st, prefix, B, P, S, rows);
}
// The beams of every user as the decode's outputs: codes [B, K, L] unpacked
// from the path keys (code of level l in byte 3 - l), scores [B, K], beam counts [B].
__global__ void write_lists_kernel(StateDev s, int B, int K, int L, int32_t* __restrict__ items,
                                   float* __restrict__ scores, int32_t* __restrict__ n_items) {
  const int total = B * K;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const uint32_t key = s.path[i];
    for (int l = 0; l < L; ++l) items[(size_t)i * L + l] = (int32_t)((key >> (8 * (3 - l))) & 0xFFu);
    scores[i] = s.score[i];
    if (i % K == 0) n_items[i / K] = s.nb[i / K];
  }
}

void launch_write_lists(const StateDev& s, int B, int K, int L, int32_t* items, float* scores, int32_t* n_items,
                        hipStream_t st) {
  const int blocks = std::max(1, std::min(1024, (B * K + 255) / 256));
  hipLaunchKernelGGL(write_lists_kernel, dim3(blocks), dim3(256), 0, st, s, B, K, L, items, scores, n_items);
}

void launch_broadcast_prefix_kv(void* pk, void* pv, int B, int H, size_t head_bytes, size_t shared_bytes,
                                hipStream_t st) {
  const size_t total = (size_t)(B - 1) * H * (shared_bytes / 16) * 2;
  const int blocks = (int)std::max<size_t>(1, std::min<size_t>(4096, (total + 255) / 256));
  hipLaunchKernelGGL(broadcast_prefix_kv_kernel, dim3(blocks), dim3(256), 0, st, (unsigned char*)pk,
                     (unsigned char*)pv, B, H, head_bytes, shared_bytes);
}
void launch_draft_beam_scores(const StateDev& s, const TreeDev& tr, const float* lpq, const float* rootq, int nitem,
                              int codebook, int L, int B, hipStream_t st) {
  hipLaunchKernelGGL(draft_beam_scores_kernel, dim3(B), dim3(64), 0, st, s, tr, lpq, rootq, nitem, codebook, L);
}
void launch_draft_select(const StateDev& s, const TreeDev& tr, const TrieDev& trie, const float* lpq,
                         const float* rootq, int nitem, int item_base, int codebook, int L, int j, int N, int* lvl_lo,
                         int* lvl_hi, unsigned long long* keys, int max_cand, int B, hipStream_t st) {
  hipLaunchKernelGGL(draft_select_kernel, dim3(B), dim3(256), 0, st, s, tr, trie, lpq, rootq, nitem, item_base,
                     codebook, L, j, N, lvl_lo, lvl_hi, keys, max_cand);
}
void launch_verify_strict(const StateDev& s, const TreeDev& tr, const TrieDev& trie, const float* lpt,
                          const float* roott, int nitem, int codebook, int L, unsigned long long* keys, int max_cand,
                          int* accepted, int* t_after, int B, hipStream_t st) {
  hipLaunchKernelGGL(verify_strict_kernel, dim3(B), dim3(256), 0, st, s, tr, trie, lpt, roott, nitem, codebook, L,
                     keys, max_cand, accepted, t_after);
}

}  // namespace atspeed
