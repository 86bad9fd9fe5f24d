// Device helpers shared by the selection kernels: path keys, selection keys,
// trie lookup, candidate generation and radix TopK (one workgroup per user).
#pragma once
#include "common.h"
#include "select.h"

namespace atspeed {

__device__ __forceinline__ uint32_t path_with(uint32_t path, int level0, int code) {
  return path | ((uint32_t)code << (8 * (3 - level0)));
}
__device__ __forceinline__ int path_code(uint32_t path, int level0) { return (path >> (8 * (3 - level0))) & 0xFF; }

__device__ __forceinline__ uint64_t make_key(float score, uint32_t path) {
  return ((uint64_t)(~float_order_key(score)) << 32) | path;
}
__device__ __forceinline__ float key_score(uint64_t key) {
  uint32_t k = ~(uint32_t)(key >> 32);
  uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
}

__device__ inline int trie_child(const TrieDev& t, int node, int code) {
  int lo = t.first[node], hi = lo + t.cnt[node] - 1;
  while (lo <= hi) {
    int mid = (lo + hi) >> 1, c = t.code[mid];
    if (c == code) return mid;
    if (c < code) lo = mid + 1; else hi = mid - 1;
  }
  return -1;
}

// ---------------------------------------------------------------- selection core
struct SelShared {
  int hist[256];
  int cum[4];
  unsigned long long prefix, mask;
  int need, done, count;
  int par_off[kMaxPar + 1];
};

// Keys of all trie-valid one-code extensions of the parents, into keys[].
// par_lp[i] is the log-prob row of parent i; codes of item level lvl0 (0-based).
__device__ inline int gen_candidates(const TrieDev& trie, int npar, const uint32_t* par_path, const float* par_score,
                              const int* par_trie, const float* const* par_lp, int lvl0, int codebook,
                              unsigned long long* keys, SelShared& sh) {
  const int tid = threadIdx.x;
  if (tid == 0) {
    int acc = 0;
    for (int i = 0; i < npar; ++i) { sh.par_off[i] = acc; acc += trie.cnt[par_trie[i]]; }
    sh.par_off[npar] = acc;
  }
  __syncthreads();
  const int n = sh.par_off[npar];
  for (int c = tid; c < n; c += blockDim.x) {
    int lo = 0, hi = npar - 1;
    while (lo < hi) {  // last parent whose offset <= c
      int mid = (lo + hi + 1) >> 1;
      if (sh.par_off[mid] <= c) lo = mid; else hi = mid - 1;
    }
    const int child = trie.first[par_trie[lo]] + (c - sh.par_off[lo]);
    const int code = trie.code[child];
    const float s = par_score[lo] + par_lp[lo][codebook * lvl0 + code];
    keys[c] = make_key(s, path_with(par_path[lo], lvl0, code));
  }
  __syncthreads();
  return n;
}

// The nsel smallest keys, ascending, into out[]; returns their number.
__device__ inline int select_smallest(const unsigned long long* keys, int n, int nsel, unsigned long long* out, SelShared& sh) {
  const int tid = threadIdx.x, nt = blockDim.x;
  if (nsel > n) nsel = n;
  if (tid == 0) { sh.prefix = 0; sh.mask = 0; sh.need = nsel; sh.done = (nsel == n); sh.count = 0; }
  __syncthreads();
  for (int shift = 56; shift >= 0 && !sh.done; shift -= 8) {
    for (int i = tid; i < 256; i += nt) sh.hist[i] = 0;
    __syncthreads();
    const unsigned long long pf = sh.prefix, mk = sh.mask;
    for (int c = tid; c < n; c += nt) {
      unsigned long long k = keys[c];
      if ((k & mk) == pf) atomicAdd(&sh.hist[(k >> shift) & 255], 1);
    }
    __syncthreads();
    if (tid < 64) {
      // wave 0 finds the bucket b where the running count first reaches need:
      // a prefix sum over 4 buckets per lane, then the one lane holding the
      // crossing (below b < need <= below b + hist[b]) records it
      const int h[4] = {sh.hist[4 * tid], sh.hist[4 * tid + 1], sh.hist[4 * tid + 2], sh.hist[4 * tid + 3]};
      const int s4 = h[0] + h[1] + h[2] + h[3];
      int incl = s4;
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (tid >= o) incl += y;
      }
      const int need = sh.need;
      int below = incl - s4, b = -1, bbelow = 0, hb = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (b < 0 && below < need && below + h[q] >= need) { b = 4 * tid + q; bbelow = below; hb = h[q]; }
        below += h[q];
      }
      if (b >= 0) {
        sh.need = need - bbelow;
        sh.prefix |= (unsigned long long)b << shift;
        sh.mask |= 0xFFull << shift;
        if (hb == need - bbelow) sh.done = 1;
      }
    }
    __syncthreads();
  }
  const unsigned long long pf = sh.prefix, mk = sh.mask;
  const bool all = (nsel == n);
  for (int c = tid; c < n; c += nt) {
    unsigned long long k = keys[c];
    if (all || (k & mk) <= pf) {
      int slot = atomicAdd(&sh.count, 1);
      if (slot < kMaxSel) out[kMaxSel + slot] = k;  // unsorted staging half
    }
  }
  __syncthreads();
  for (int i = tid; i < nsel; i += nt) {
    unsigned long long k = out[kMaxSel + i];
    int rank = 0;
    for (int j = 0; j < nsel; ++j) rank += out[kMaxSel + j] < k;
    out[rank] = k;
  }
  __syncthreads();
  return nsel;
}

}  // namespace atspeed
