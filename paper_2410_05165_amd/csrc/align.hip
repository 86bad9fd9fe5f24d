// Draft alignment (Sec. 3.1 AtSpeed-S, Sec. 3.2 AtSpeed-R) on the device: the
// training contexts of a batch, the per-context loss and its gradient with
// respect to the draft's item logits, the gradient of the draft's item head, and
// the optimizer step.
//
// A training context c is a user's root (the last prefix position) or a prefix
// y_<t (1 <= t < L) of one of the user's training sequences; its weight w counts
// the sequences through it over (|y| x users), the aggregation of the Align
// losses.  q and p are the draft's and the target's item-token distributions at
// c, V_c the K trie-valid codes of the next level with the largest q (ties: the
// smaller code).
//   S: l = sum_{v in V_c} q_v (log p_K - log p_v)  (the reverse KL over V_c minus
//      the density regulariser; the q log q terms cancel), with p_K the target's
//      probability of the K-th sequence's code at this level;
//      dl/dz_j = q_j (a_j [j in V_c] - l), a_v = log p_K - log p_v;
//   R: l = TVD(p', q') over V_c (both renormalised to V_c);
//      dl/dz_j = [j in V_c] q'_j (s_j - sum_v s_v q'_v) / 2, s_v = sign(q'_v - p'_v).
// V_c is held fixed in the gradient (the selection is piecewise constant in z).
#include <algorithm>
#include "common.h"
#include "kernels.h"
#include "select_dev.h"

namespace atspeed {

// Key of the depth-`depth` prefix of a path key.
__device__ __forceinline__ uint32_t key_prefix(uint32_t key, int depth) {
  return depth <= 0 ? 0u : depth >= 4 ? key : key & ~(0xFFFFFFFFu >> (8 * depth));
}

// Context tree of one batch: per user, every distinct prefix of depth 1..L of its
// n training sequences (items [u][k][0..len_k), len_k = lens[u][k] or L),
// level-ordered.  ctx_weight of a node: sum of 1 / (|y| B) over the sequences
// it is a proper prefix of (its weight as a context; the root's in
// root_weight); label_weight: the same over the sequences it is a prefix of
// (its weight as the label of its parent context).  kslot[u][t] = tree slot of
// the last sequence's depth-t prefix (1 <= t < L).  Flags err (and leaves the
// user an empty tree) when n is outside 1..S, a length outside 1..L, the last
// sequence shorter than L, a prefix outside the catalog or more nodes than
// max_nodes.
__global__ void align_tree_kernel(const int* __restrict__ items, const int* __restrict__ lens,
                                  const int* __restrict__ n_items, int S, TreeDev tr, TrieDev trie, int B, int L,
                                  int item_base, int codebook, float* __restrict__ ctx_weight,
                                  float* __restrict__ label_weight, float* __restrict__ root_weight,
                                  int* __restrict__ kslot, int* err) {
  const int u = blockIdx.x;
  if (threadIdx.x != 0) return;
  const size_t tb = (size_t)u * tr.max_nodes;
  const int n = n_items[u];
  tr.n_nodes[u] = 0;
  root_weight[u] = 0.f;
  for (int i = 0; i < tr.max_nodes; ++i) {
    ctx_weight[tb + i] = 0.f;
    label_weight[tb + i] = 0.f;
  }
  for (int t = 0; t < L; ++t) kslot[u * L + t] = -1;
  bool ok = n >= 1 && n <= S;
  for (int k = 0; ok && k < n; ++k) {
    const int len = lens ? lens[u * S + k] : L;
    ok = len >= 1 && len <= L && (k < n - 1 || len == L);
    int node = 0;
    for (int l = 0; ok && l < len; ++l) {
      const int code = items[((size_t)u * S + k) * L + l];
      ok = code >= 0 && code < codebook;
      if (ok) node = trie_child(trie, node, code);
      ok = ok && node >= 0;
    }
  }
  int cnt = 0;
  float rw = 0.f;
  for (int l = 1; ok && l <= L; ++l)
    for (int k = 0; ok && k < n; ++k) {
      const int len = lens ? lens[u * S + k] : L;
      if (len < l) continue;
      const float wy = 1.f / (float)(len * B);
      if (l == 1) rw += wy;
      const int* y = items + ((size_t)u * S + k) * L;
      uint32_t key = 0;
      for (int i = 0; i < l; ++i) key = path_with(key, i, y[i]);
      int found = -1, parent = -1;
      for (int i = 0; i < cnt; ++i) {
        if (tr.depth[tb + i] == l && tr.tpath[tb + i] == key) found = i;
        if (l > 1 && tr.depth[tb + i] == l - 1 && tr.tpath[tb + i] == key_prefix(key, l - 1)) parent = i;
      }
      if (found < 0) {
        if (cnt == tr.max_nodes) {
          ok = false;
          break;
        }
        const int ptrie = parent >= 0 ? tr.ttrie[tb + parent] : 0;
        tr.token[tb + cnt] = item_base + codebook * (l - 1) + y[l - 1];
        tr.parent[tb + cnt] = parent;
        tr.depth[tb + cnt] = l;
        tr.q_score[tb + cnt] = 0.f;
        tr.tpath[tb + cnt] = key;
        tr.ttrie[tb + cnt] = trie_child(trie, ptrie, y[l - 1]);
        found = cnt++;
      }
      label_weight[tb + found] += wy;
      if (len > l) ctx_weight[tb + found] += wy;
      if (k == n - 1 && l < L) kslot[u * L + l] = (int)tb + found;   // tree slot u * max_nodes + s
    }
  if (!ok) {
    atomicOr(err, 4);
    return;
  }
  tr.n_nodes[u] = cnt;
  root_weight[u] = rw;
}

// log p_K of every level: the target's log-prob of the last sequence's t-th code
// at its own prefix (the root's row at t = 0).
__global__ void align_logpk_kernel(const int* __restrict__ items, const int* __restrict__ n_items,
                                   const int* __restrict__ kslot, const float* __restrict__ lp,
                                   const float* __restrict__ root, int S, int L, int codebook, int nitem,
                                   float* __restrict__ log_pK) {
  const int u = blockIdx.x, t = threadIdx.x;
  if (t >= L) return;
  const int n = n_items[u];
  if (n < 1 || n > S || (t > 0 && kslot[u * L + t] < 0)) {
    log_pK[u * L + t] = 0.f;
    return;
  }
  const int code = items[((size_t)u * S + n - 1) * L + t];
  const float* row = t == 0 ? root + (size_t)u * nitem : lp + (size_t)kslot[u * L + t] * nitem;
  log_pK[u * L + t] = row[codebook * t + code];
}

// One workgroup per context row: rows [0, B) are the users' roots, row B + r is
// row r of the draft's forward over the context tree.  dz row = alpha w dl/dz +
// (1 - alpha)(w q - lw), lw the label weights of the context's children in the
// tree (the next codes of the sequences through it); loss row = alpha w l +
// (1 - alpha)(-sum_children lw log q).
__global__ void __launch_bounds__(256)
align_grad_kernel(AlignRows ar, TrieDev trie, TreeDev tr, int B, int nitem, int codebook, int L, int K, int mode,
                  float alpha, float* __restrict__ dz, float* __restrict__ loss_rows) {
  __shared__ float cq[256], cp[256], chw[256];
  __shared__ int ccol[256], sel[256];
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  if (row >= B + *ar.Mdev) return;
  int u, slot, node, lvl;
  if (row < B) {
    u = row;
    slot = -1;
    node = 0;
    lvl = 0;
  } else {
    u = ar.user[row - B];
    slot = ar.slot[row - B];   // u * max_nodes + local slot
    node = tr.ttrie[slot];
    lvl = tr.depth[slot];
  }
  const size_t tb = (size_t)u * tr.max_nodes;
  const float w = slot < 0 ? ar.root_weight[u] : ar.ctx_weight[slot];
  const float* lq = slot < 0 ? ar.lq_root + (size_t)u * nitem : ar.lq + (size_t)slot * nitem;
  const float* lp = slot < 0 ? ar.lp_root + (size_t)u * nitem : ar.lp + (size_t)slot * nitem;
  float* g = dz + (size_t)row * nitem;
  const int n = lvl < L ? trie.cnt[node] : 0;
  if (!(w > 0.f) || n == 0) {
    for (int j = tid; j < nitem; j += 256) g[j] = 0.f;
    if (tid == 0) loss_rows[row] = 0.f;
    return;
  }
  // candidates: the trie children of the context's node (codes of level lvl);
  // labels: the label weight of the context's tree child with each code
  const int first = trie.first[node];
  if (tid < n) {
    const int col = codebook * lvl + trie.code[first + tid];
    ccol[tid] = col;
    cq[tid] = lq[col];
    cp[tid] = lp[col];
  }
  if (tid < codebook) chw[tid] = 0.f;
  __syncthreads();
  const int nn = tr.n_nodes[u];
  for (int i = tid; i < nn; i += 256) {
    const bool child = slot < 0 ? tr.depth[tb + i] == 1 : tr.parent[tb + i] == (int)(slot - tb);
    if (child) chw[path_code(tr.tpath[tb + i], lvl)] = ar.label_weight[tb + i];
  }
  // V_c: rank by (q desc, column asc) below K
  const int kk = min(K, n);
  if (tid < n) {
    int r = 0;
    for (int i = 0; i < n; ++i) r += (cq[i] > cq[tid]) || (cq[i] == cq[tid] && ccol[i] < ccol[tid]);
    sel[tid] = r < kk;
  }
  __syncthreads();
  // sums in a fixed order (one thread)
  if (tid == 0) {
    float l = 0.f, sq = 0.f, sp = 0.f, sg = 0.f, rec = 0.f;
    const float lpk = mode == 0 ? ar.log_pK[u * L + lvl] : 0.f;
    if (mode == 0) {
      for (int i = 0; i < n; ++i)
        if (sel[i]) l += expf(cq[i]) * (lpk - cp[i]);
    } else {
      for (int i = 0; i < n; ++i)
        if (sel[i]) {
          sq += expf(cq[i]);
          sp += expf(cp[i]);
        }
      for (int i = 0; i < n; ++i)
        if (sel[i]) {
          const float qn = expf(cq[i]) / sq, pn = expf(cp[i]) / sp;
          l += 0.5f * fabsf(pn - qn);
          sg += (qn > pn ? 1.f : (qn < pn ? -1.f : 0.f)) * qn;
        }
    }
    for (int c = 0; c < codebook; ++c)
      if (chw[c] != 0.f) rec -= chw[c] * lq[codebook * lvl + c];
    red[0] = l;
    red[1] = mode == 0 ? lpk : sq;
    red[2] = sp;
    red[3] = sg;
    loss_rows[row] = alpha * w * l + (1.f - alpha) * rec;
  }
  __syncthreads();
  const float l = red[0];
  // every column: the align term outside V_c plus the recommendation term's w q
  for (int j = tid; j < nitem; j += 256) {
    const float q = expf(lq[j]);
    g[j] = (mode == 0 ? alpha * (-w * q * l) : 0.f) + (1.f - alpha) * w * q;
  }
  __syncthreads();
  if (tid < n && sel[tid]) {
    const float q = expf(cq[tid]);
    if (mode == 0) {
      g[ccol[tid]] += alpha * w * q * (red[1] - cp[tid]);
    } else {
      const float sq = red[1], sp = red[2], sg = red[3];
      const float qn = q / sq, pn = expf(cp[tid]) / sp;
      const float sgn = qn > pn ? 1.f : (qn < pn ? -1.f : 0.f);
      g[ccol[tid]] += alpha * w * 0.5f * qn * (sgn - sg);
    }
  }
  __syncthreads();
  if (tid < codebook && chw[tid] != 0.f) g[codebook * lvl + tid] -= (1.f - alpha) * chw[tid];
}

// dW[v][k] = sum_rows dz[row][v] * h[row][k] in fp32; rows [0, B) take the
// roots' hidden states, the others the context rows'.  A 64x64 output tile per
// workgroup (4x4 per thread), rows in a fixed order, so the result does not
// depend on the launch.
template <class T>
__global__ void __launch_bounds__(256)
head_grad_kernel(const float* __restrict__ dz, const T* __restrict__ h_root, const T* __restrict__ h_rows,
                 const int* __restrict__ Mdev, int B, int nitem, int d, float* __restrict__ dW) {
  __shared__ float Gs[32][65];
  __shared__ float Hs[32][65];
  const int v0 = blockIdx.y * 64, k0 = blockIdx.x * 64, tid = threadIdx.x;
  const int nrows = B + *Mdev;
  const int tv = tid / 16, tk = tid % 16;
  float acc[4][4] = {};
  for (int r0 = 0; r0 < nrows; r0 += 32) {
    for (int i = tid; i < 32 * 64; i += 256) {
      const int r = i / 64, c = i % 64, row = r0 + r;
      float gv = 0.f, hv = 0.f;
      if (row < nrows) {
        if (v0 + c < nitem) gv = dz[(size_t)row * nitem + v0 + c];
        if (k0 + c < d)
          hv = row < B ? St<T>::ld(h_root + (size_t)row * d + k0 + c)
                       : St<T>::ld(h_rows + (size_t)(row - B) * d + k0 + c);
      }
      Gs[r][c] = gv;
      Hs[r][c] = hv;
    }
    __syncthreads();
    for (int r = 0; r < 32; ++r) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = Gs[r][tv + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Hs[r][tk + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int v = v0 + tv + 16 * i, k = k0 + tk + 16 * j;
      if (v < nitem && k < d) dW[(size_t)v * d + k] = acc[i][j];
    }
}

// The hidden states the head gradient used, fp32: roots at rows [0, B), the
// context rows at B + their tree slot.
template <class T>
__global__ void align_hidden_kernel(const T* __restrict__ h_root, const T* __restrict__ h_rows,
                                    const int* __restrict__ slot, const int* __restrict__ Mdev, int B, int d,
                                    float* __restrict__ out) {
  const int row = blockIdx.x;
  if (row >= B + *Mdev) return;
  const T* src = row < B ? h_root + (size_t)row * d : h_rows + (size_t)(row - B) * d;
  float* dst = out + (size_t)(row < B ? row : B + slot[row - B]) * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) dst[k] = St<T>::ld(src + k);
}

// AdamW on the fp32 master copy (decoupled weight decay), then the head the
// draft reads (rounded to its dtype).
template <class T>
__global__ void adamw_kernel(float* __restrict__ master, float* __restrict__ m, float* __restrict__ v,
                             const float* __restrict__ g, T* __restrict__ head, size_t n, float lr, float b1,
                             float b2, float eps, float wd, float c1, float c2) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const float gi = g[i];
    const float mi = b1 * m[i] + (1.f - b1) * gi, vi = b2 * v[i] + (1.f - b2) * gi * gi;
    m[i] = mi;
    v[i] = vi;
    float w = master[i];
    w -= lr * wd * w;
    w -= lr * (mi / c1) / (sqrtf(vi / c2) + eps);
    master[i] = w;
    St<T>::st(head + i, w);
  }
}

// log((1 - lam) q + lam p) in place over the draft's log-prob rows: rows
// [0, nrows[u]) of each user's rows_per_user (every row when nrows is null).
// lam 1 and 0 copy one model's row unchanged.
__global__ void __launch_bounds__(256)
mix_logprobs_kernel(float* __restrict__ lq, const float* __restrict__ lp, const int* __restrict__ nrows,
                    int rows_per_user, int nitem, float lam) {
  const int u = blockIdx.x / rows_per_user, r = blockIdx.x % rows_per_user;
  if (nrows && r >= nrows[u]) return;
  const size_t off = (size_t)blockIdx.x * nitem;
  for (int j = threadIdx.x; j < nitem; j += 256) {
    const float q = lq[off + j], p = lp[off + j];
    float m;
    if (lam >= 1.f) {
      m = p;
    } else if (lam <= 0.f) {
      m = q;
    } else {
      const float mx = fmaxf(q, p);
      m = mx + logf((1.f - lam) * expf(q - mx) + lam * expf(p - mx));
    }
    lq[off + j] = m;
  }
}

void launch_mix_logprobs(float* lq, const float* lp, const int* nrows, int B, int rows_per_user, int nitem, float lam,
                         hipStream_t st) {
  hipLaunchKernelGGL(mix_logprobs_kernel, dim3(B * rows_per_user), dim3(256), 0, st, lq, lp, nrows, rows_per_user,
                     nitem, lam);
}

void launch_align_tree(const int* items, const int* lens, const int* n_items, int S, const TreeDev& tr,
                       const TrieDev& trie, int B, int L, int item_base, int codebook, float* ctx_weight,
                       float* label_weight, float* root_weight, int* kslot, int* err, hipStream_t st) {
  hipLaunchKernelGGL(align_tree_kernel, dim3(B), dim3(64), 0, st, items, lens, n_items, S, tr, trie, B, L, item_base,
                     codebook, ctx_weight, label_weight, root_weight, kslot, err);
}

void launch_align_logpk(const int* items, const int* n_items, const int* kslot, const float* lp, const float* root,
                        int B, int S, int L, int codebook, int nitem, float* log_pK, hipStream_t st) {
  hipLaunchKernelGGL(align_logpk_kernel, dim3(B), dim3(64), 0, st, items, n_items, kslot, lp, root, S, L, codebook,
                     nitem, log_pK);
}

void launch_align_grad(const AlignRows& ar, const TrieDev& trie, const TreeDev& tr, int B, int M, int nitem,
                       int codebook, int L, int K, int mode, float alpha, float* dz, float* loss_rows,
                       hipStream_t st) {
  hipLaunchKernelGGL(align_grad_kernel, dim3(B + M), dim3(256), 0, st, ar, trie, tr, B, nitem, codebook, L, K, mode,
                     alpha, dz, loss_rows);
}

void launch_head_grad(bool bf16, const float* dz, const void* h_root, const void* h_rows, const int* Mdev, int B,
                      int nitem, int d, float* dW, hipStream_t st) {
  const dim3 grid((d + 63) / 64, (nitem + 63) / 64);
  if (bf16)
    hipLaunchKernelGGL(head_grad_kernel<bf16_t>, grid, dim3(256), 0, st, dz, (const bf16_t*)h_root,
                       (const bf16_t*)h_rows, Mdev, B, nitem, d, dW);
  else
    hipLaunchKernelGGL(head_grad_kernel<float>, grid, dim3(256), 0, st, dz, (const float*)h_root,
                       (const float*)h_rows, Mdev, B, nitem, d, dW);
}

void launch_align_hidden(bool bf16, const void* h_root, const void* h_rows, const int* slot, const int* Mdev, int B,
                         int M, int d, float* out, hipStream_t st) {
  if (bf16)
    hipLaunchKernelGGL(align_hidden_kernel<bf16_t>, dim3(B + M), dim3(256), 0, st, (const bf16_t*)h_root,
                       (const bf16_t*)h_rows, slot, Mdev, B, d, out);
  else
    hipLaunchKernelGGL(align_hidden_kernel<float>, dim3(B + M), dim3(256), 0, st, (const float*)h_root,
                       (const float*)h_rows, slot, Mdev, B, d, out);
}

void launch_adamw(bool bf16, float* master, float* m, float* v, const float* g, void* head, size_t n, float lr,
                  float b1, float b2, float eps, float wd, int step, hipStream_t st) {
  const float c1 = 1.f - powf(b1, (float)step), c2 = 1.f - powf(b2, (float)step);
  const int blocks = (int)std::min<size_t>(2048, (n + 255) / 256);
  if (bf16)
    hipLaunchKernelGGL(adamw_kernel<bf16_t>, dim3(blocks), dim3(256), 0, st, master, m, v, g, (bf16_t*)head, n, lr, b1,
                       b2, eps, wd, c1, c2);
  else
    hipLaunchKernelGGL(adamw_kernel<float>, dim3(blocks), dim3(256), 0, st, master, m, v, g, (float*)head, n, lr, b1,
                       b2, eps, wd, c1, c2);
}

}  // namespace atspeed
