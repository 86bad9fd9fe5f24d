// Tree attention (tree-based attention of Sec. 3.3 and its implementation
// appendix, restated): a query row of user u attends to the first nctx keys of
// u's prefix KV cache and to its own tree keys (ancestors and itself, at most L).
// The same kernel runs causal prefill (nctx = position + 1, no tree keys).
//
// One workgroup handles (user, head, 64 query rows of that user): the user's
// prefix K/V are streamed once per workgroup in 64-key tiles through LDS and
// shared by all its queries (the prefix is read once per user per layer, not
// once per tree token).  Softmax is online (running max and sum) in fp32.
#include "common.h"
#include "kernels.h"

namespace atspeed {

constexpr int AQ = 64;  // query rows per workgroup
constexpr int AK = 64;  // keys per tile

template <class T, int DH>
__global__ void __launch_bounds__(256)
attn_kernel(const T* __restrict__ q, const T* __restrict__ pk, const T* __restrict__ pv,
            const T* __restrict__ tk, const T* __restrict__ tv, T* __restrict__ out, Rows rows,
            int H, int Pmax, float qscale) {
  constexpr int DP = DH + 1;
  constexpr int OD = DH / 16;  // output dims per thread
  extern __shared__ __align__(16) float sm[];
  float* Qs = sm;                  // [AQ][DP]
  float* Ks = Qs + AQ * DP;        // [AK][DP]
  float* Vs = Ks + AK * DP;        // [AK][DH]
  float* Ss = Vs + AK * DH;        // [AQ][AK + 1]
  __shared__ float m_s[AQ], l_s[AQ], a_s[AQ];
  __shared__ int nctx_s[AQ], anc_s[AQ][4], nanc_s[AQ];
  __shared__ int kmax_s;

  const int u = blockIdx.y, h = blockIdx.x;
  const int ubeg = rows.user_off[u], uend = rows.user_off[u + 1];
  const int r0 = ubeg + blockIdx.z * AQ;
  if (r0 >= uend) return;
  const int nq = min(AQ, uend - r0);
  const int tid = threadIdx.x;
  const int d = H * DH;

  if (tid == 0) kmax_s = 0;
  __syncthreads();
  if (tid < AQ) {
    int n = 0;
    if (tid < nq) {
      n = rows.nctx[r0 + tid];
      nanc_s[tid] = rows.nanc[r0 + tid];
      for (int a = 0; a < 4; ++a) anc_s[tid][a] = rows.anc[(r0 + tid) * 4 + a];
    } else {
      nanc_s[tid] = 0;
    }
    nctx_s[tid] = n;
    m_s[tid] = -INFINITY;
    l_s[tid] = 0.f;
    atomicMax(&kmax_s, n);
  }
  for (int i = tid; i < AQ * DH; i += 256) {
    int r = i / DH, c = i % DH;
    Qs[r * DP + c] = r < nq ? St<T>::ld(q + (size_t)(r0 + r) * d + h * DH + c) * qscale : 0.f;
  }
  __syncthreads();
  const int kmax = kmax_s;

  const int tq = tid >> 4, tkk = tid & 15;   // S tile: 4 queries x 4 keys per thread
  const int oq = tid >> 4, od = tid & 15;    // O tile: 4 queries x OD dims per thread
  float o[4][OD];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < OD; ++j) o[i][j] = 0.f;

  const size_t kvbase = ((size_t)u * H + h) * Pmax * DH;
  for (int k0 = 0; k0 < kmax; k0 += AK) {
    const int nk = min(AK, kmax - k0);
    for (int i = tid; i < AK * DH; i += 256) {
      int r = i / DH, c = i % DH;
      float kv = 0.f, vv = 0.f;
      if (r < nk) {
        kv = St<T>::ld(pk + kvbase + (size_t)(k0 + r) * DH + c);
        vv = St<T>::ld(pv + kvbase + (size_t)(k0 + r) * DH + c);
      }
      Ks[r * DP + c] = kv;
      Vs[r * DH + c] = vv;
    }
    __syncthreads();
    float s[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) s[i][j] = 0.f;
    for (int c = 0; c < DH; ++c) {
      float qa[4], ka[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) qa[i] = Qs[(tq * 4 + i) * DP + c];
#pragma unroll
      for (int j = 0; j < 4; ++j) ka[j] = Ks[(tkk + 16 * j) * DP + c];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) s[i][j] += qa[i] * ka[j];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int qi = tq * 4 + i, kj = tkk + 16 * j;
        Ss[qi * (AK + 1) + kj] = (k0 + kj < nctx_s[qi]) ? s[i][j] : -INFINITY;
      }
    __syncthreads();
    {  // online softmax: 4 threads per query row, 16 keys each
      const int row = tid >> 2, part = tid & 3;
      float mx = -INFINITY;
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, Ss[row * (AK + 1) + part * 16 + j]);
      mx = fmaxf(mx, __shfl_xor(mx, 1));
      mx = fmaxf(mx, __shfl_xor(mx, 2));
      const float mold = m_s[row];
      const float mnew = fmaxf(mold, mx);
      float sum = 0.f;
      for (int j = 0; j < 16; ++j) {
        float sv = Ss[row * (AK + 1) + part * 16 + j];
        float p = (sv == -INFINITY) ? 0.f : exp2f(sv - mnew);
        Ss[row * (AK + 1) + part * 16 + j] = p;
        sum += p;
      }
      sum += __shfl_xor(sum, 1);
      sum += __shfl_xor(sum, 2);
      __syncthreads();  // every lane has read m_s[row] before it changes
      if (part == 0) {
        const float alpha = (mold == -INFINITY) ? 0.f : exp2f(mold - mnew);
        a_s[row] = alpha;
        l_s[row] = l_s[row] * alpha + sum;
        m_s[row] = mnew;
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float al = a_s[oq * 4 + i];
#pragma unroll
      for (int j = 0; j < OD; ++j) o[i][j] *= al;
    }
    for (int kj = 0; kj < nk; ++kj) {
      float pa[4], va[OD];
#pragma unroll
      for (int i = 0; i < 4; ++i) pa[i] = Ss[(oq * 4 + i) * (AK + 1) + kj];
#pragma unroll
      for (int j = 0; j < OD; ++j) va[j] = Vs[kj * DH + od + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < OD; ++j) o[i][j] += pa[i] * va[j];
    }
    __syncthreads();
  }

  if (tk != nullptr) {  // tree keys: ancestors and self of every query
    {
      const int row = tid >> 2, a = tid & 3;
      float sv = -INFINITY;
      if (a < nanc_s[row]) {
        const T* kp = tk + (size_t)anc_s[row][a] * d + h * DH;
        float acc = 0.f;
        for (int c = 0; c < DH; ++c) acc += Qs[row * DP + c] * St<T>::ld(kp + c);
        sv = acc;
      }
      float mx = sv;
      mx = fmaxf(mx, __shfl_xor(mx, 1));
      mx = fmaxf(mx, __shfl_xor(mx, 2));
      const float mold = m_s[row];
      const float mnew = fmaxf(mold, mx);
      const float p = (sv == -INFINITY) ? 0.f : exp2f(sv - mnew);
      Ss[row * (AK + 1) + a] = p;
      float sum = p;
      sum += __shfl_xor(sum, 1);
      sum += __shfl_xor(sum, 2);
      __syncthreads();
      if (a == 0) {
        const float alpha = (mold == -INFINITY) ? 0.f : exp2f(mold - mnew);
        a_s[row] = alpha;
        l_s[row] = l_s[row] * alpha + sum;
        m_s[row] = mnew;
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qi = oq * 4 + i;
      const float al = a_s[qi];
#pragma unroll
      for (int j = 0; j < OD; ++j) o[i][j] *= al;
      for (int a = 0; a < nanc_s[qi]; ++a) {
        const float p = Ss[qi * (AK + 1) + a];
        const T* vp = tv + (size_t)anc_s[qi][a] * d + h * DH;
#pragma unroll
        for (int j = 0; j < OD; ++j) o[i][j] += p * St<T>::ld(vp + od + 16 * j);
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int qi = oq * 4 + i;
    if (qi >= nq) continue;
    const float inv = 1.f / l_s[qi];
#pragma unroll
    for (int j = 0; j < OD; ++j) St<T>::st(out + (size_t)(r0 + qi) * d + h * DH + od + 16 * j, o[i][j] * inv);
  }
}

// ---------------------------------------------------------------- bf16 MFMA kernel
// Per workgroup: (head, user, 64 query rows); wave w owns queries 16w..16w+15.
// S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (A = K rows from LDS, B = Q from
// registers): lane l holds S^T[key 4g+i][query l%16] (g = l/16) of each 16-key
// block, so the probabilities of its query sit in registers in exactly the
// B-operand layout of O^T = V^T P^T, with the 32 keys of a k-step ordered
// {4g..4g+3, 16+4g..16+4g+3} on both operands.  V^T is staged transposed in LDS.
// Each query's tree keys (ancestors and itself) follow, one dot product split
// over the 4 lanes of the query.
template <int DH>
__global__ void __launch_bounds__(256)
attn_mfma_kernel(const bf16_t* __restrict__ q, const bf16_t* __restrict__ pk, const bf16_t* __restrict__ pv,
                 const bf16_t* __restrict__ tk, const bf16_t* __restrict__ tv, bf16_t* __restrict__ out, Rows rows,
                 int H, int Pmax, float qscale, int nusers, int nqblk) {
  constexpr int KT = 64;          // keys per tile
  constexpr int NKS = DH / 32;    // k-steps of S^T
  constexpr int NDB = DH / 16;    // 16-dim blocks of O^T
  constexpr int CPR = DH / 8;     // 16-byte chunks per K row
  __shared__ __align__(16) bf16_t Ks[KT * DH];
  __shared__ __align__(16) bf16_t Vt[DH * KT];
  __shared__ int kmax_s;

  // Workgroup L runs on XCD L % 8.  The Z query blocks of one (user, head) pair
  // get consecutive indices on one XCD, so they run together and share the
  // pair's prefix tiles in that XCD's L2; the pairs are dealt round-robin over
  // the XCDs.
  const int Lw = blockIdx.x, xcd = Lw & 7, qi8 = Lw >> 3, Z = nqblk;
  const int pair = (qi8 / Z) * 8 + xcd, zb = qi8 % Z;
  if (pair >= H * nusers) return;
  const int u = pair / H, h = pair % H;
  const int ubeg = rows.user_off[u], uend = rows.user_off[u + 1];
  const int r0 = ubeg + zb * 64;
  if (r0 >= uend) return;
  const int nq = min(64, uend - r0);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, ql = lane & 15;
  const int qi = wave * 16 + ql;
  const bool valid = qi < nq;
  const int row = r0 + (valid ? qi : 0);
  const int d = H * DH;

  if (tid == 0) kmax_s = 0;
  __syncthreads();
  const int nctx = valid ? rows.nctx[row] : 0;
  if (g == 0) atomicMax(&kmax_s, nctx);

  bf16x8_t qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    if (valid) qf[ks] = *reinterpret_cast<const bf16x8_t*>(q + (size_t)row * d + h * DH + ks * 32 + g * 8);
    else qf[ks] = bf16x8_t{};
  }
  f32x4_t o[NDB];
#pragma unroll
  for (int i = 0; i < NDB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, lsum = 0.f;
  __syncthreads();
  const int kmax = kmax_s;
  const size_t kvbase = ((size_t)u * H + h) * Pmax * DH;

  // Tile staging: K rows as 16-byte chunks (NKC per thread); V transposed, each
  // thread taking 4 consecutive keys x 8 dims so that it writes 8-byte runs of
  // 4 keys per dim.  The next tile's global loads are issued into registers
  // before the current tile's matrix work, so their latency hides behind it.
  constexpr int NKC = KT * CPR / 256;
  const bool vthr = tid < 16 * CPR;
  const int vkg = tid / CPR, vj = tid % CPR;
  u32x4_t kreg[NKC], vreg[4];
  auto fetch = [&](int k0) {
    const int nk = min(KT, kmax - k0);
#pragma unroll
    for (int c = 0; c < NKC; ++c) {
      const int idx = tid + c * 256, key = idx / CPR, j = idx % CPR;
      kreg[c] = key < nk ? *reinterpret_cast<const u32x4_t*>(pk + kvbase + (size_t)(k0 + key) * DH + j * 8)
                         : u32x4_t{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = 4 * vkg + i;
      vreg[i] = vthr && key < nk ? *reinterpret_cast<const u32x4_t*>(pv + kvbase + (size_t)(k0 + key) * DH + vj * 8)
                                 : u32x4_t{0u, 0u, 0u, 0u};
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int c = 0; c < NKC; ++c) {
      const int idx = tid + c * 256, key = idx / CPR, j = idx % CPR;
      *reinterpret_cast<u32x4_t*>(Ks + key * DH + ((j ^ (key & (CPR - 1))) * 8)) = kreg[c];
    }
    if (vthr) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int dim = vj * 8 + e, sh = (e & 1) * 16;
        uint2 w;
        w.x = ((vreg[0][e >> 1] >> sh) & 0xffffu) | (((vreg[1][e >> 1] >> sh) & 0xffffu) << 16);
        w.y = ((vreg[2][e >> 1] >> sh) & 0xffffu) | (((vreg[3][e >> 1] >> sh) & 0xffffu) << 16);
        *reinterpret_cast<uint2*>(Vt + dim * KT + ((vkg ^ (dim & 15)) << 2)) = w;
      }
    }
  };
  if (kmax > 0) fetch(0);
  for (int k0 = 0; k0 < kmax; k0 += KT) {
    stash();
    __syncthreads();
    if (k0 + KT < kmax) fetch(k0 + KT);
    // S^T for 4 blocks of 16 keys
    f32x4_t sc[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      sc[kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const int key = kb * 16 + ql;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const int j = ks * 4 + g;
        const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(Ks + key * DH + ((j ^ (key & (CPR - 1))) * 8));
        sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], sc[kb], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = k0 + kb * 16 + g * 4 + i;
        const float v = key < nctx ? sc[kb][i] * qscale : -INFINITY;
        sc[kb][i] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m, mx);
    const float alpha = (m == -INFINITY) ? 0.f : exp2f(m - mnew);
    float ps = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = (sc[kb][i] == -INFINITY) ? 0.f : exp2f(sc[kb][i] - mnew);
        sc[kb][i] = p;
        ps += p;
      }
    lsum = lsum * alpha + ps;
    m = mnew;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] *= alpha;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      // P as the sum of two bf16 parts (hi + lo ~ 16 significant bits), so the
      // probabilities keep near-fp32 precision through the bf16 MFMA.
      bf16x8_t pf, pl;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pf[i] = (__bf16)sc[2 * kk][i];
        pf[4 + i] = (__bf16)sc[2 * kk + 1][i];
        pl[i] = (__bf16)(sc[2 * kk][i] - (float)pf[i]);
        pl[4 + i] = (__bf16)(sc[2 * kk + 1][i] - (float)pf[4 + i]);
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int dim = db * 16 + ql;
        const int c0 = ((kk * 8 + g) ^ (dim & 15)) << 2, c1 = ((kk * 8 + 4 + g) ^ (dim & 15)) << 2;
        const uint2 lo = *reinterpret_cast<const uint2*>(Vt + dim * KT + c0);
        const uint2 hi = *reinterpret_cast<const uint2*>(Vt + dim * KT + c1);
        u32x4_t w4 = {lo.x, lo.y, hi.x, hi.y};
        bf16x8_t vf = __builtin_bit_cast(bf16x8_t, w4);
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[db], 0, 0, 0);
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl, o[db], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  if (tk != nullptr && valid) {  // tree keys: ancestors and self
    const int na = rows.nanc[row];
    int slot[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) slot[a] = a < na ? rows.anc[row * 4 + a] : 0;
    float sa[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      float part = 0.f;
      if (a < na) {
        const bf16_t* kp = tk + (size_t)slot[a] * d + h * DH;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(kp + ks * 32 + g * 8);
#pragma unroll
          for (int e = 0; e < 8; ++e) part += (float)qf[ks][e] * (float)kf[e];
        }
      }
      part += __shfl_xor(part, 16);
      part += __shfl_xor(part, 32);
      sa[a] = a < na ? part * qscale : -INFINITY;
    }
    float mx = fmaxf(fmaxf(sa[0], sa[1]), fmaxf(sa[2], sa[3]));
    const float mnew = fmaxf(m, mx);
    const float alpha = (m == -INFINITY) ? 0.f : exp2f(m - mnew);
    float ps = 0.f;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      sa[a] = a < na ? exp2f(sa[a] - mnew) : 0.f;
      ps += sa[a];
    }
    lsum = lsum * alpha + (g == 0 ? ps : 0.f);
    m = mnew;
    // lane (query, g) holds dims db*16 + 4g .. +3 of O: one 8-byte load per
    // (ancestor, block), the blocks of one ancestor issued together
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] *= alpha;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      if (a < na) {
        const bf16_t* vp = tv + (size_t)slot[a] * d + h * DH + g * 4;
        uint2 vw[NDB];
#pragma unroll
        for (int db = 0; db < NDB; ++db) vw[db] = *reinterpret_cast<const uint2*>(vp + db * 16);
        const float p = sa[a];
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          o[db][0] += p * __uint_as_float(vw[db].x << 16);
          o[db][1] += p * __uint_as_float(vw[db].x & 0xffff0000u);
          o[db][2] += p * __uint_as_float(vw[db].y << 16);
          o[db][3] += p * __uint_as_float(vw[db].y & 0xffff0000u);
        }
      }
    }
  }
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (valid) {
    const float inv = 1.f / lsum;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      uint2 w;
      w.x = (uint32_t)f2bf(o[db][0] * inv) | ((uint32_t)f2bf(o[db][1] * inv) << 16);
      w.y = (uint32_t)f2bf(o[db][2] * inv) | ((uint32_t)f2bf(o[db][3] * inv) << 16);
      *reinterpret_cast<uint2*>(out + (size_t)row * d + h * DH + db * 16 + g * 4) = w;
    }
  }
}

template <int DH>
static hipError_t launch_attn_mfma(const AttnCall& a, hipStream_t st) {
  const float qscale = 1.4426950408889634f / sqrtf((float)DH);
  // one-dimensional grid: ceil(pairs / 8) groups of 8 pairs x Z query blocks
  const int Z = std::max(1, (a.Tq + 63) / 64);
  const long pairs = (long)a.H * a.B;
  const long nwg = (pairs + 7) / 8 * 8 * Z;
  if (nwg > 0x7fffffffL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(attn_mfma_kernel<DH>, dim3((unsigned)nwg), dim3(256), 0, st, (const bf16_t*)a.q,
                     (const bf16_t*)a.pk, (const bf16_t*)a.pv, (const bf16_t*)a.tk, (const bf16_t*)a.tv,
                     (bf16_t*)a.out, a.rows, a.H, a.Pmax, qscale, a.B, Z);
  return hipGetLastError();
}

template <class T, int DH>
static hipError_t launch_attn(const AttnCall& a, hipStream_t st) {
  constexpr int DP = DH + 1;
  const size_t smem = sizeof(float) * (AQ * DP + AK * DP + AK * DH + AQ * (AK + 1));
  auto kern = attn_kernel<T, DH>;
  // set on every launch: the attribute is per device, and this path (fp32
  // workloads) is not the one whose launch cost matters
  hipError_t err = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  if (err != hipSuccess) return err;
  const float qscale = 1.4426950408889634f / sqrtf((float)DH);  // log2(e) / sqrt(d_head)
  dim3 grid(a.H, a.B, (a.Tq + AQ - 1) / AQ);  // query blocks slowest, as in the MFMA kernel
  hipLaunchKernelGGL(kern, grid, dim3(256), smem, st, (const T*)a.q, (const T*)a.pk, (const T*)a.pv,
                     (const T*)a.tk, (const T*)a.tv, (T*)a.out, a.rows, a.H, a.Pmax, qscale);
  return hipGetLastError();
}

hipError_t attention(const AttnCall& a, hipStream_t st) {
  if (a.bf16) {
    if (a.dh == 64) return launch_attn_mfma<64>(a, st);
    if (a.dh == 128) return launch_attn_mfma<128>(a, st);
  } else {
    if (a.dh == 64) return launch_attn<float, 64>(a, st);
    if (a.dh == 128) return launch_attn<float, 128>(a, st);
    if (a.dh == 32) return launch_attn<float, 32>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace atspeed
