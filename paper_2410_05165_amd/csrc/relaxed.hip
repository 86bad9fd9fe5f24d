// Relaxed sampling verification (Sec. 3.2, Eq. 6, Algorithm 2) on the device:
// sampled drafting and the per-user acceptance / residual resampling.
//
// Level distributions: for parent beams S and a model M, pi_M(c) is
// exp(S_M(c)/tau) normalised over the trie-valid extensions ext(S), with S_M the
// cumulative log-prob.  Two readings of Algorithm 2 (the paper's listing is not
// self-consistent):
//   EXACT  K slots per level, each drawn from pi_q (Gumbel-max); slot k accepted
//          iff log u_k <= log pi_p(y_k) - log pi_q(y_k); a rejected slot is
//          redrawn from norm(max(0, pi_p - pi_q)); the level's beams are the
//          distinct slots; the step stops at the first level with a rejection.
//   PAPER  N distinct drafts per level (Gumbel-top-N over pi_q); each accepted by
//          the same test with pi_p over ext(T_{j-1}) (zero outside); >= K accepted
//          -> K kept uniformly at random (Gumbel-top-K of equal weights), level
//          accepted; else K - #accepted distinct redraws from the residual with
//          the accepted zeroed, and the step stops.
// Randomness: Philox4x32-10 (Salmon et al., SC'11), key = the context seed,
// counter (user, step, level*2^16 + draw, cand*4 + tag), tags 0 draft, 1 accept,
// 2 subset, 3 target draw / residual; cand = lexicographic rank of the parent
// among the level's parents * codebook + code (0 for per-draw uniforms);
// u = ((x0 >> 9) + 0.5) * 2^-23, Gumbel g = -log(-log u).
#include "common.h"
#include "select.h"
#include "select_dev.h"

namespace atspeed {

__device__ inline uint32_t philox_x0(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0, n1 = (uint32_t)p1;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1, n3 = (uint32_t)p0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c0;
}
__device__ inline float philox_u(const RelaxArgs& ra, int u, int step, int lvl, int draw, int cand, int tag) {
  const uint32_t x = philox_x0((uint32_t)u, (uint32_t)step, (uint32_t)(lvl * 65536 + draw), (uint32_t)(cand * 4 + tag),
                               ra.k0, ra.k1);
  return ((float)(x >> 9) + 0.5f) * (1.0f / 8388608.0f);
}
__device__ inline float philox_g(const RelaxArgs& ra, int u, int step, int lvl, int draw, int cand, int tag) {
  return -logf(-logf(philox_u(ra, u, step, lvl, draw, cand, tag)));
}

__device__ inline float bmax(float v, float* red) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}
__device__ inline float bsum(float v, float* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}
__device__ inline unsigned long long bmin64(unsigned long long v, unsigned long long* red) {
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long w = __shfl_xor(v, o);
    v = w < v ? w : v;
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  unsigned long long m = red[0];
  for (int i = 1; i < 4; ++i) m = red[i] < m ? red[i] : m;
  return m;
}

// Parents of a level, in LDS.  rank = lexicographic rank of the path.
struct Parents {
  uint32_t path[kMaxPar];
  float sp[kMaxPar], sq[kMaxPar];
  int trie[kMaxPar], slot[kMaxPar], rank[kMaxPar];
  const float* lpp[kMaxPar];
  const float* lpq[kMaxPar];
  int n;
};

__device__ inline void rank_parents(Parents& P) {
  for (int i = threadIdx.x; i < P.n; i += blockDim.x) {
    int r = 0;
    for (int q = 0; q < P.n; ++q) r += P.path[q] < P.path[i];
    P.rank[i] = r;
  }
  __syncthreads();
}

// Extensions of the parents: path, parent index, canonical index, target and
// draft cumulative scores (target only when the parent has a target row).
__device__ inline int expand(const TrieDev& trie, const Parents& P, int lvl0, int codebook, CandBuf cb, SelShared& sh) {
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int i = 0; i < P.n; ++i) { sh.par_off[i] = acc; acc += trie.cnt[P.trie[i]]; }
    sh.par_off[P.n] = acc;
  }
  __syncthreads();
  const int n = sh.par_off[P.n];
  for (int c = threadIdx.x; c < n; c += blockDim.x) {
    int lo = 0, hi = P.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (sh.par_off[mid] <= c) lo = mid; else hi = mid - 1;
    }
    const int child = trie.first[P.trie[lo]] + (c - sh.par_off[lo]);
    const int code = trie.code[child];
    const int col = codebook * lvl0 + code;
    cb.path[c] = path_with(P.path[lo], lvl0, code);
    cb.par[c] = lo;
    cb.cidx[c] = P.rank[lo] * codebook + code;
    cb.sp[c] = P.lpp[lo] ? P.sp[lo] + P.lpp[lo][col] : -INFINITY;
    cb.sq[c] = P.lpq[lo] ? P.sq[lo] + P.lpq[lo][col] : -INFINITY;
  }
  __syncthreads();
  return n;
}

// log-sum-exp of v[0..n)/tau (block-wide).
__device__ inline float block_lse(const float* v, int n, float tau, float* red) {
  float m = -INFINITY;
  for (int c = threadIdx.x; c < n; c += blockDim.x) m = fmaxf(m, v[c] / tau);
  m = bmax(m, red);
  float s = 0.f;
  for (int c = threadIdx.x; c < n; c += blockDim.x) s += expf(v[c] / tau - m);
  s = bsum(s, red);
  return m + logf(s);
}

// Position of each wanted path among the level's candidates (the first match,
// -1 if none), by the whole block: each thread compares its share of the
// candidates with every wanted path (want and idx in LDS), where one thread per
// wanted path would walk thousands of candidates in global memory.
__device__ inline void find_candidates(const uint32_t* want, int nwant, const uint32_t* cpath, int n, int* idx) {
  for (int i = threadIdx.x; i < nwant; i += blockDim.x) idx[i] = INT_MAX;
  __syncthreads();
  for (int c = threadIdx.x; c < n; c += blockDim.x) {
    const uint32_t p = cpath[c];
    for (int i = 0; i < nwant; ++i)
      if (want[i] == p) atomicMin(&idx[i], c);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nwant; i += blockDim.x)
    if (idx[i] == INT_MAX) idx[i] = -1;
  __syncthreads();
}

// The same for the tree nodes of depth lvl (first matching node, -1 if none).
__device__ inline void find_nodes(const uint32_t* want, int nwant, const uint32_t* tpath, const int* depth, int lvl,
                                  int ntree, int* idx) {
  for (int i = threadIdx.x; i < nwant; i += blockDim.x) idx[i] = INT_MAX;
  __syncthreads();
  for (int t = threadIdx.x; t < ntree; t += blockDim.x) {
    if (depth[t] != lvl) continue;
    const uint32_t p = tpath[t];
    for (int i = 0; i < nwant; ++i)
      if (want[i] == p) atomicMin(&idx[i], t);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nwant; i += blockDim.x)
    if (idx[i] == INT_MAX) idx[i] = -1;
  __syncthreads();
}

// ---------------------------------------------------------------- drafting
// One drafted level (relaxed modes): EXACT draws K slots, PAPER N distinct.
// New nodes are appended to the tree; lvl_lo/lvl_hi bound them; zq records the
// draft's normaliser of this level; slot_node maps EXACT slots to nodes.
__global__ void __launch_bounds__(256)
draft_relaxed_kernel(StateDev s, TreeDev tr, TrieDev trie, const float* lpq, const float* rootq, int nitem,
                     int item_base, int codebook, int L, int j, int* lvl_lo, int* lvl_hi, CandBuf cball,
                     int max_cand, RelaxArgs ra) {
  __shared__ Parents P;
  __shared__ SelShared sh;
  __shared__ unsigned long long sel[2 * kMaxSel];
  __shared__ unsigned long long red64[4];
  __shared__ float red[4];
  __shared__ uint32_t win[kMaxSel];
  __shared__ int winslot[kMaxSel];
  const int u = blockIdx.x, tid = threadIdx.x;
  const int t = s.t[u];
  const int J = min(s.gamma, L - t);
  const size_t tb = (size_t)u * tr.max_nodes;
  if (t >= L || j > J) {
    if (tid == 0) { lvl_lo[u] = tr.n_nodes[u]; lvl_hi[u] = tr.n_nodes[u]; }
    return;
  }
  const int lvl = t + j, lvl0 = lvl - 1, step = s.steps[u];
  if (j == 1) {
    P.n = t == 0 ? 1 : s.nb[u];
    for (int i = tid; i < P.n; i += blockDim.x) {
      if (t == 0) { P.path[i] = 0; P.sq[i] = 0.f; P.trie[i] = 0; P.slot[i] = -1; P.lpq[i] = rootq + (size_t)u * nitem; }
      else {
        const int sl = s.beam_slot[u * s.K + i];
        P.path[i] = s.path[u * s.K + i]; P.sq[i] = s.qscore[u * s.K + i]; P.trie[i] = s.trie[u * s.K + i];
        P.slot[i] = sl; P.lpq[i] = lpq + (tb + sl) * nitem;
      }
      P.lpp[i] = nullptr;
      P.sp[i] = 0.f;
    }
  } else {
    const int a = lvl_lo[u];
    P.n = lvl_hi[u] - a;
    for (int i = tid; i < P.n; i += blockDim.x) {
      const int sl = a + i;
      P.path[i] = tr.tpath[tb + sl]; P.sq[i] = tr.q_score[tb + sl]; P.trie[i] = tr.ttrie[tb + sl];
      P.slot[i] = sl; P.lpq[i] = lpq + (tb + sl) * nitem; P.lpp[i] = nullptr; P.sp[i] = 0.f;
    }
  }
  __syncthreads();
  rank_parents(P);
  CandBuf cb = cball.offset((size_t)u * max_cand);
  const int n = expand(trie, P, lvl0, codebook, cb, sh);
  const float zq = block_lse(cb.sq, n, ra.tau, red);
  if (tid == 0) ra.zq[u * (L + 1) + lvl] = zq;
  const int base = tr.n_nodes[u];
  int nnew;
  if (ra.mode == 1) {  // EXACT: K i.i.d. slots, then their distinct set in lexicographic order
    const int K = s.K;
    for (int k = 0; k < K; ++k) {
      unsigned long long best = ~0ull;
      for (int c = tid; c < n; c += blockDim.x) {
        const float v = cb.sq[c] / ra.tau + philox_g(ra, u, step, lvl, k, cb.cidx[c], 0);
        const unsigned long long key = make_key(v, cb.path[c]);
        best = key < best ? key : best;
      }
      best = bmin64(best, red64);
      if (tid == 0) win[k] = (uint32_t)best;
    }
    __syncthreads();
    if (tid == 0) {
      int m = 0;
      for (int k = 0; k < K; ++k) {  // insertion into the sorted distinct list
        int pos = 0;
        while (pos < m && (uint32_t)sel[pos] < win[k]) ++pos;
        if (pos < m && (uint32_t)sel[pos] == win[k]) continue;
        for (int q = m; q > pos; --q) sel[q] = sel[q - 1];
        sel[pos] = win[k];
        ++m;
      }
      for (int k = 0; k < K; ++k) {
        int pos = 0;
        while ((uint32_t)sel[pos] != win[k]) ++pos;
        winslot[k] = base + pos;
        ra.slot_node[((size_t)u * (L + 1) + lvl) * K + k] = base + pos;
      }
      sh.count = m;
    }
    __syncthreads();
    nnew = sh.count;
  } else {  // PAPER: N distinct by Gumbel-top-N, in draw order
    unsigned long long* keys = ra.keys + (size_t)u * max_cand;
    for (int c = tid; c < n; c += blockDim.x) {
      const float v = cb.sq[c] / ra.tau + philox_g(ra, u, step, lvl, 0, cb.cidx[c], 0);
      keys[c] = make_key(v, cb.path[c]);
    }
    __syncthreads();
    nnew = select_smallest(keys, n, ra.N, sel, sh);
  }
  for (int i = tid; i < nnew; i += blockDim.x) {
    const uint32_t path = (uint32_t)sel[i];
    const int code = path_code(path, lvl0);
    const uint32_t ppre = lvl0 == 0 ? 0u : (path & ~(0xFFFFFFFFu >> (8 * lvl0)));
    int pi = 0;
    for (int q = 0; q < P.n; ++q) if (P.path[q] == ppre) { pi = q; break; }
    const int sl = base + i;
    tr.token[tb + sl] = item_base + codebook * lvl0 + code;
    tr.parent[tb + sl] = P.slot[pi];
    tr.depth[tb + sl] = lvl;
    tr.q_score[tb + sl] = P.sq[pi] + P.lpq[pi][codebook * lvl0 + code];
    tr.tpath[tb + sl] = path;
    tr.ttrie[tb + sl] = trie_child(trie, P.trie[pi], code);
  }
  __syncthreads();
  if (tid == 0) {
    tr.n_nodes[u] = base + nnew;
    lvl_lo[u] = base;
    lvl_hi[u] = base + nnew;
  }
}

// ---------------------------------------------------------------- verification
__global__ void __launch_bounds__(256)
verify_relaxed_kernel(StateDev s, TreeDev tr, TrieDev trie, const float* lpt, const float* roott, const float* lpq,
                      const float* rootq, int nitem, int codebook, int L, CandBuf cball, int max_cand, RelaxArgs ra,
                      int* accepted_out, int* t_after_out) {
  __shared__ Parents P;
  __shared__ SelShared sh;
  __shared__ unsigned long long sel[2 * kMaxSel];
  __shared__ unsigned long long red64[4];
  __shared__ float red[4];
  __shared__ uint32_t fin[kMaxSel];      // per-slot / per-draft outcome paths
  __shared__ int acc_flag[kMaxSel];
  __shared__ int nacc_s;
  __shared__ uint32_t want[kMaxSel];     // paths looked up among the candidates / tree nodes
  __shared__ int cand_of[kMaxSel], node_of[kMaxSel];
  __shared__ int run_s[2];               // first node of a depth and the end of its run
  const int u = blockIdx.x, tid = threadIdx.x;
  const int t = s.t[u], K = s.K;
  if (t >= L) {
    if (tid == 0) { if (accepted_out) accepted_out[u] = -1; if (t_after_out) t_after_out[u] = t; }
    return;
  }
  const size_t tb = (size_t)u * tr.max_nodes;
  const int J = min(s.gamma, L - t), step = s.steps[u];
  const int ntree = tr.n_nodes[u];
  // T_0 = Y_t with target and draft scores
  P.n = t == 0 ? 1 : s.nb[u];
  for (int i = tid; i < P.n; i += blockDim.x) {
    if (t == 0) {
      P.path[i] = 0; P.sp[i] = 0.f; P.sq[i] = 0.f; P.trie[i] = 0; P.slot[i] = -1;
      P.lpp[i] = roott + (size_t)u * nitem; P.lpq[i] = rootq + (size_t)u * nitem;
    } else {
      const int sl = s.beam_slot[u * K + i];
      P.path[i] = s.path[u * K + i]; P.sp[i] = s.score[u * K + i]; P.sq[i] = s.qscore[u * K + i];
      P.trie[i] = s.trie[u * K + i]; P.slot[i] = sl;
      P.lpp[i] = lpt + (tb + sl) * nitem; P.lpq[i] = lpq + (tb + sl) * nitem;
    }
  }
  __syncthreads();
  CandBuf cb = cball.offset((size_t)u * max_cand);
  unsigned long long* keys = ra.keys + (size_t)u * max_cand;
  int accepted = 0, t_after = t, nout = 0;
  for (int j = 1; j <= J + 1; ++j) {
    const int lvl = t + j, lvl0 = lvl - 1;
    if (lvl > L) break;
    const bool bonus = j == J + 1;
    rank_parents(P);
    const int n = expand(trie, P, lvl0, codebook, cb, sh);
    const float zp = block_lse(cb.sp, n, ra.tau, red);
    const float zq = ra.mode == 1 ? block_lse(cb.sq, n, ra.tau, red) : ra.zq[u * (L + 1) + lvl];
    int ok = 1;
    if (bonus) {
      // next level straight from pi_p (EXACT: K slots; PAPER: Gumbel-top-K)
      if (ra.mode == 1) {
        for (int k = 0; k < K; ++k) {
          unsigned long long best = ~0ull;
          for (int c = tid; c < n; c += blockDim.x) {
            const float v = cb.sp[c] / ra.tau - zp + philox_g(ra, u, step, lvl, k, cb.cidx[c], 3);
            const unsigned long long key = make_key(v, cb.path[c]);
            best = key < best ? key : best;
          }
          best = bmin64(best, red64);
          if (tid == 0) fin[k] = (uint32_t)best;
        }
        if (tid == 0) nout = K;
      } else {
        for (int c = tid; c < n; c += blockDim.x)
          keys[c] = make_key(cb.sp[c] / ra.tau - zp + philox_g(ra, u, step, lvl, 0, cb.cidx[c], 3), cb.path[c]);
        __syncthreads();
        const int m = select_smallest(keys, n, K, sel, sh);
        for (int i = tid; i < m; i += blockDim.x) fin[i] = (uint32_t)sel[i];
        if (tid == 0) nout = m;
      }
    } else if (ra.mode == 1) {  // EXACT
      if (tid == 0) nacc_s = 0;
      __syncthreads();
      for (int k = tid; k < K; k += blockDim.x)
        want[k] = tr.tpath[tb + ra.slot_node[((size_t)u * (L + 1) + lvl) * K + k]];
      __syncthreads();
      find_candidates(want, K, cb.path, n, cand_of);
      for (int k = tid; k < K; k += blockDim.x) {
        const uint32_t y = want[k];
        const int ci = cand_of[k];
        float a = -INFINITY;
        if (ci >= 0) a = (cb.sp[ci] / ra.tau - zp) - (cb.sq[ci] / ra.tau - zq);
        const bool acc = logf(philox_u(ra, u, step, lvl, k, 0, 1)) <= a;
        acc_flag[k] = acc;
        fin[k] = y;
        if (acc) atomicAdd(&nacc_s, 1);
      }
      __syncthreads();
      ok = nacc_s == K;
      if (!ok) {
        for (int k = 0; k < K; ++k) {
          if (acc_flag[k]) continue;  // uniform across the block (LDS)
          unsigned long long best = ~0ull;
          for (int c = tid; c < n; c += blockDim.x) {
            const float r = expf(cb.sp[c] / ra.tau - zp) - expf(cb.sq[c] / ra.tau - zq);
            if (r > 0.f) {
              const unsigned long long key = make_key(logf(r) + philox_g(ra, u, step, lvl, k, cb.cidx[c], 3), cb.path[c]);
              best = key < best ? key : best;
            }
          }
          best = bmin64(best, red64);
          if (tid == 0 && best != ~0ull) fin[k] = (uint32_t)best;
          __syncthreads();
        }
      }
      if (tid == 0) nout = K;
    } else {  // PAPER: drafted nodes of this level, in draw order
      if (tid == 0) { nacc_s = 0; }
      __syncthreads();
      // the drafted nodes of this level: the run of depth lvl that starts at its
      // first node (the tree is level-ordered)
      if (tid == 0) { run_s[0] = ntree; run_s[1] = ntree; }
      __syncthreads();
      for (int i = tid; i < ntree; i += blockDim.x)
        if (tr.depth[tb + i] == lvl) atomicMin(&run_s[0], i);
      __syncthreads();
      const int d0 = run_s[0];
      for (int i = d0 + tid; i < ntree; i += blockDim.x)
        if (tr.depth[tb + i] != lvl) atomicMin(&run_s[1], i);
      __syncthreads();
      const int d1 = run_s[1];
      const int nd = min(d1 - d0, kMaxSel);
      for (int i = tid; i < nd; i += blockDim.x) want[i] = tr.tpath[tb + d0 + i];
      __syncthreads();
      find_candidates(want, nd, cb.path, n, cand_of);
      for (int i = tid; i < nd; i += blockDim.x) {
        const int ci = cand_of[i];
        float a = -INFINITY;
        if (ci >= 0) a = (cb.sp[ci] / ra.tau - zp) - (tr.q_score[tb + d0 + i] / ra.tau - zq);
        const bool acc = logf(philox_u(ra, u, step, lvl, i, 0, 1)) <= a;
        acc_flag[i] = acc;
        if (acc) atomicAdd(&nacc_s, 1);
      }
      __syncthreads();
      const int na = nacc_s;
      ok = na >= K;
      // keys of the accepted drafts: K of them uniformly (equal-weight Gumbel), or all of them
      for (int i = tid; i < nd; i += blockDim.x)
        keys[i] = acc_flag[i] ? make_key(ok ? philox_g(ra, u, step, lvl, i, 0, 2) : 0.f, tr.tpath[tb + d0 + i]) : ~0ull;
      __syncthreads();
      const int m = select_smallest(keys, nd, ok ? K : na, sel, sh);
      for (int i = tid; i < m; i += blockDim.x) fin[i] = (uint32_t)sel[i];
      __syncthreads();
      int mo = m;
      if (!ok) {
        // residual over ext(T_{j-1}) with the accepted drafts zeroed, Gumbel-top-(K - accepted)
        float qz;
        for (int c = tid; c < n; c += blockDim.x) {
          bool zero = false;
          for (int q = 0; q < m; ++q) zero |= (uint32_t)sel[q] == cb.path[c];
          qz = cb.sq[c] / ra.tau - zq;
          const float r = zero ? 0.f : expf(cb.sp[c] / ra.tau - zp) - expf(qz);
          keys[c] = r > 0.f ? make_key(logf(r) + philox_g(ra, u, step, lvl, 0, cb.cidx[c], 3), cb.path[c]) : ~0ull;
        }
        // number of positive residuals (each thread counts the keys it wrote;
        // held in a register, so select_smallest may reuse sh.count)
        float cnt = 0.f;
        for (int c = tid; c < n; c += blockDim.x) cnt += keys[c] != ~0ull ? 1.f : 0.f;
        const int npos = (int)bsum(cnt, red);
        __syncthreads();
        const int extra = select_smallest(keys, n, min(K - m, npos), sel, sh);
        for (int i = tid; i < extra; i += blockDim.x) fin[m + i] = (uint32_t)sel[i];
        mo = m + extra;
      }
      if (tid == 0) nout = mo;
    }
    __syncthreads();
    // T_j: distinct outcomes, lexicographic; parents of the next level
    if (tid == 0) {
      int m = 0;
      for (int k = 0; k < nout; ++k) {
        int pos = 0;
        while (pos < m && (uint32_t)sel[pos] < fin[k]) ++pos;
        if (pos < m && (uint32_t)sel[pos] == fin[k]) continue;
        for (int q = m; q > pos; --q) sel[q] = sel[q - 1];
        sel[pos] = fin[k];
        ++m;
      }
      sh.count = m;
    }
    __syncthreads();
    const int m = sh.count;
    for (int i = tid; i < m; i += blockDim.x) want[i] = (uint32_t)sel[i];
    __syncthreads();
    find_candidates(want, m, cb.path, n, cand_of);
    find_nodes(want, m, tr.tpath + tb, tr.depth + tb, lvl, ntree, node_of);
    uint32_t mp = 0; float msp = 0.f, msq = 0.f; int mtrie = -1, mslot = -1;
    if (tid < m) {
      mp = want[tid];
      const int ci = cand_of[tid] >= 0 ? cand_of[tid] : 0;  // every outcome is a candidate
      const int pi = cb.par[ci];
      msp = cb.sp[ci];
      mtrie = trie_child(trie, P.trie[pi], path_code(mp, lvl0));
      mslot = node_of[tid];
      msq = mslot >= 0 ? tr.q_score[tb + mslot] : cb.sq[ci];
    }
    __syncthreads();
    if (tid < m) {
      P.path[tid] = mp; P.sp[tid] = msp; P.sq[tid] = msq; P.trie[tid] = mtrie; P.slot[tid] = mslot;
      P.lpp[tid] = mslot >= 0 ? lpt + (tb + mslot) * nitem : nullptr;
      P.lpq[tid] = mslot >= 0 ? lpq + (tb + mslot) * nitem : nullptr;
    }
    if (tid == 0) P.n = m;
    __syncthreads();
    if (bonus) { accepted = J; t_after = lvl; break; }
    if (lvl == L) { accepted = ok ? j : j - 1; t_after = L; break; }
    if (!ok) { accepted = j - 1; t_after = lvl; break; }
  }
  for (int i = tid; i < P.n; i += blockDim.x) {
    s.path[u * K + i] = P.path[i];
    s.score[u * K + i] = P.sp[i];
    s.trie[u * K + i] = P.trie[i];
  }
  if (tid == 0) {
    s.nb[u] = P.n;
    s.t[u] = t_after;
    s.steps[u] += 1;
    if (accepted_out) accepted_out[u] = accepted;
    if (t_after_out) t_after_out[u] = t_after;
  }
}

void launch_draft_relaxed(const StateDev& s, const TreeDev& tr, const TrieDev& trie, const float* lpq,
                          const float* rootq, int nitem, int item_base, int codebook, int L, int j, int* lvl_lo,
                          int* lvl_hi, const CandBuf& cb, int max_cand, const RelaxArgs& ra, int B, hipStream_t st) {
  hipLaunchKernelGGL(draft_relaxed_kernel, dim3(B), dim3(256), 0, st, s, tr, trie, lpq, rootq, nitem, item_base,
                     codebook, L, j, lvl_lo, lvl_hi, cb, max_cand, ra);
}

void launch_verify_relaxed(const StateDev& s, const TreeDev& tr, const TrieDev& trie, const float* lpt,
                           const float* roott, const float* lpq, const float* rootq, int nitem, int codebook, int L,
                           const CandBuf& cb, int max_cand, const RelaxArgs& ra, int* accepted, int* t_after, int B,
                           hipStream_t st) {
  hipLaunchKernelGGL(verify_relaxed_kernel, dim3(B), dim3(256), 0, st, s, tr, trie, lpt, roott, lpq, rootq, nitem,
                     codebook, L, cb, max_cand, ra, accepted, t_after);
}

}  // namespace atspeed
