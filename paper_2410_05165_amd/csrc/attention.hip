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

  const int u = blockIdx.z, h = blockIdx.y;
  const int ubeg = rows.user_off[u], uend = rows.user_off[u + 1];
  const int r0 = ubeg + blockIdx.x * AQ;
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

template <class T, int DH>
static hipError_t launch_attn(const AttnCall& a, hipStream_t st) {
  constexpr int DP = DH + 1;
  const size_t smem = sizeof(float) * (AQ * DP + AK * DP + AK * DH + AQ * (AK + 1));
  auto kern = attn_kernel<T, DH>;
  static bool attr = false;
  if (!attr) {
    hipError_t err = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (err != hipSuccess) return err;
    attr = true;
  }
  const float qscale = 1.4426950408889634f / sqrtf((float)DH);  // log2(e) / sqrt(d_head)
  dim3 grid((a.Tq + AQ - 1) / AQ, a.H, a.B);
  hipLaunchKernelGGL(kern, grid, dim3(256), smem, st, (const T*)a.q, (const T*)a.pk, (const T*)a.pv,
                     (const T*)a.tk, (const T*)a.tv, (T*)a.out, a.rows, a.H, a.Pmax, qscale);
  return hipGetLastError();
}

hipError_t attention(const AttnCall& a, hipStream_t st) {
  if (a.bf16) {
    if (a.dh == 64) return launch_attn<bf16_t, 64>(a, st);
    if (a.dh == 128) return launch_attn<bf16_t, 128>(a, st);
    if (a.dh == 32) return launch_attn<bf16_t, 32>(a, st);
  } else {
    if (a.dh == 64) return launch_attn<float, 64>(a, st);
    if (a.dh == 128) return launch_attn<float, 128>(a, st);
    if (a.dh == 32) return launch_attn<float, 32>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace atspeed
