// Dense projections of the decoder block: Y[M, N] = X[M, K] · W[N, K]^T.
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16 (fp32 accumulate), block tile
// BM x BN x 64 staged through LDS (double buffer, XOR-swizzled 16-byte chunks),
// wave tile TM x TN blocks of 32x32.  Epilogues are fused:
//   QKV   rotary embedding on q and k (rotate-half pairs sit in registers of the
//         same lane: partner block tn ^ (d_head/64)), rounding to bf16, q to its
//         row buffer, k/v scattered into the prefix cache or the tree KV buffer;
//   GU    gate and up columns share a tile (first/second half of each wave's
//         blocks), out = bf16(SiLU(gate) * up);
//   RESID residual stream x += acc (fp32);
//   STORE fp32 logits.
// M is read from device memory (the tree size is only known on the device);
// tiles past it exit at once.
//
// fp32 path (fp32 workloads): plain LDS-tiled FMA GEMM to a scratch matrix,
// then an elementwise epilogue kernel with the same semantics.
#include "common.h"
#include "kernels.h"

namespace atspeed {

enum { EPI_STORE = 0, EPI_RESID = 1, EPI_GU = 2, EPI_QKV = 3 };
enum { BMAP_PLAIN = 0, BMAP_QKV = 1, BMAP_GU = 2 };

struct EpiArgs {
  float* out;        // STORE: [M, ldo] fp32; RESID: residual [M, ldo] fp32
  int ldo;
  bf16_t* hout;      // GU: [M, f] bf16
  // QKV
  bf16_t* q;         // [M, d]
  bf16_t* kdst;      // prefix cache or tree KV base of this layer
  bf16_t* vdst;
  const float* cosT; // [max_pos, dh/2]
  const float* sinT;
  Rows rows;
  int kv_mode;       // 0 prefix cache [B][H][Pmax][dh], 1 tree [slot][d]
  int Pmax;
  int d, dh, H;
};

struct BArgs {
  const bf16_t* w0;
  const bf16_t* w1;
  const bf16_t* w2;
  int split;         // QKV: d; GU: f
};

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

template <int WM, int WN, int TM, int TN>
struct Tile {
  static constexpr int NT = 64 * WM * WN;
  static constexpr int BM = WM * TM * 32;
  static constexpr int BN = WN * TN * 32;
  static constexpr int BK = 64;
  static constexpr int A_CH = BM * 8 / NT;  // 16-byte chunks per thread per stage
  static constexpr int B_CH = BN * 8 / NT;
  static constexpr int A_BYTES = BM * 128;
  static constexpr int B_BYTES = BN * 128;
  static constexpr int STAGE = A_BYTES + B_BYTES;
};

template <int WM, int WN, int TM, int TN, int BMAP, int EPI>
__global__ void __launch_bounds__(64 * WM * WN)
gemm_bf16_kernel(const bf16_t* __restrict__ A, int lda, const int* __restrict__ Mdev, int N, int K,
                 BArgs b, EpiArgs e) {
  using T = Tile<WM, WN, TM, TN>;
  extern __shared__ __align__(16) unsigned char smem[];
  const int M = *Mdev;
  const int tile_m = blockIdx.y, tile_n = blockIdx.x;
  const int m0 = tile_m * T::BM;
  if (m0 >= M) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wave_m = wave / WN, wave_n = wave % WN;

  // global -> register staging: 16-byte chunk offsets (uint4 units) from a base
  // pointer.  A tile lies in one matrix for PLAIN/QKV (d % BN == 0 is checked on
  // the host); for GU the chunk's block picks the gate or the up matrix.
  const u32x4_t* a_base = reinterpret_cast<const u32x4_t*>(A);
  int a_off[T::A_CH], b_off[T::B_CH];
  bool b_hi[T::B_CH];
#pragma unroll
  for (int i = 0; i < T::A_CH; ++i) {
    int ci = tid + i * T::NT, r = ci >> 3, c = ci & 7;
    int gr = m0 + r;
    gr = gr < M ? gr : M - 1;
    a_off[i] = gr * (lda >> 3) + c;
  }
  const u32x4_t* b_base0;
  const u32x4_t* b_base1 = nullptr;
  {
    const int n_first = tile_n * T::BN;
    if (BMAP == BMAP_QKV) {
      const int which = n_first / b.split;
      b_base0 = reinterpret_cast<const u32x4_t*>(which == 0 ? b.w0 : (which == 1 ? b.w1 : b.w2));
    } else if (BMAP == BMAP_GU) {
      b_base0 = reinterpret_cast<const u32x4_t*>(b.w0);
      b_base1 = reinterpret_cast<const u32x4_t*>(b.w1);
    } else {
      b_base0 = reinterpret_cast<const u32x4_t*>(b.w0);
    }
  }
#pragma unroll
  for (int i = 0; i < T::B_CH; ++i) {
    int ci = tid + i * T::NT, r = ci >> 3, c = ci & 7;
    int row;
    b_hi[i] = false;
    if (BMAP == BMAP_GU) {
      constexpr int half = TN / 2;
      int wn = r / (TN * 32), blk = (r / 32) % TN, cc = r % 32;
      row = tile_n * (T::BN / 2) + wn * (half * 32) + (blk % half) * 32 + cc;
      row = row < b.split ? row : b.split - 1;
      b_hi[i] = blk >= half;
    } else {
      row = tile_n * T::BN + r;
      row = row < N ? row : N - 1;
      if (BMAP == BMAP_QKV) row -= (tile_n * T::BN / b.split) * b.split;
    }
    b_off[i] = row * (K >> 3) + c;
  }

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  u32x4_t ra[T::A_CH], rb[T::B_CH];
  const int nk = K / T::BK;
  int adst[T::A_CH], bdst[T::B_CH];
#pragma unroll
  for (int i = 0; i < T::A_CH; ++i) {
    int ci = tid + i * T::NT, r = ci >> 3, c = ci & 7;
    adst[i] = r * 128 + ((c ^ (r & 7)) << 4);
  }
#pragma unroll
  for (int i = 0; i < T::B_CH; ++i) {
    int ci = tid + i * T::NT, r = ci >> 3, c = ci & 7;
    bdst[i] = T::A_BYTES + r * 128 + ((c ^ (r & 7)) << 4);
  }

#pragma unroll
  for (int i = 0; i < T::A_CH; ++i) ra[i] = a_base[a_off[i]];
#pragma unroll
  for (int i = 0; i < T::B_CH; ++i) rb[i] = (BMAP == BMAP_GU && b_hi[i] ? b_base1 : b_base0)[b_off[i]];
#pragma unroll
  for (int i = 0; i < T::A_CH; ++i) *reinterpret_cast<u32x4_t*>(smem + adst[i]) = ra[i];
#pragma unroll
  for (int i = 0; i < T::B_CH; ++i) *reinterpret_cast<u32x4_t*>(smem + bdst[i]) = rb[i];
  __syncthreads();
  const int fr = lane & 31, fc = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) {
      const int ko = (kt + 1) * 8;
#pragma unroll
      for (int i = 0; i < T::A_CH; ++i) ra[i] = a_base[a_off[i] + ko];
#pragma unroll
      for (int i = 0; i < T::B_CH; ++i) rb[i] = (BMAP == BMAP_GU && b_hi[i] ? b_base1 : b_base0)[b_off[i] + ko];
    }
    const unsigned char* base = smem + (kt & 1) * T::STAGE;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8_t af[TM], bfr[TN];
      const int ch = kk * 2 + fc;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        int r = wave_m * TM * 32 + i * 32 + fr;
        af[i] = *reinterpret_cast<const bf16x8_t*>(base + r * 128 + ((ch ^ (r & 7)) << 4));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        int r = wave_n * TN * 32 + j * 32 + fr;
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(base + T::A_BYTES + r * 128 + ((ch ^ (r & 7)) << 4));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      unsigned char* nb = smem + ((kt + 1) & 1) * T::STAGE;
#pragma unroll
      for (int i = 0; i < T::A_CH; ++i) *reinterpret_cast<u32x4_t*>(nb + adst[i]) = ra[i];
#pragma unroll
      for (int i = 0; i < T::B_CH; ++i) *reinterpret_cast<u32x4_t*>(nb + bdst[i]) = rb[i];
    }
    __syncthreads();
  }

  // ---- epilogue.  acc[i][j][r] is row (r/4)*8 + (lane/32)*4 + r%4, column lane%32 of block (i, j).
  const int row0 = m0 + wave_m * TM * 32;
  const int col0 = tile_n * T::BN + wave_n * TN * 32;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = row0 + i * 32 + (r >> 2) * 8 + fc * 4 + (r & 3);
      if (row >= M) continue;
      if (EPI == EPI_STORE || EPI == EPI_RESID) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          int col = col0 + j * 32 + fr;
          if (col < N) {
            float* p = e.out + (size_t)row * e.ldo + col;
            if (EPI == EPI_STORE) *p = acc[i][j][r];
            else *p += acc[i][j][r];
          }
        }
      } else if (EPI == EPI_GU) {
        constexpr int half = TN / 2;
#pragma unroll
        for (int j = 0; j < half; ++j) {
          int fcol = tile_n * (T::BN / 2) + wave_n * (half * 32) + j * 32 + fr;
          if (fcol < b.split)
            e.hout[(size_t)row * b.split + fcol] = f2bf(silu(acc[i][j][r]) * acc[i][j + half][r]);
        }
      } else {  // EPI_QKV
        const int pos = e.rows.pos[row];
        const int halfdh = e.dh >> 1;
        const int pb = halfdh >> 5;  // partner block distance (1 for d_head 64, 2 for 128)
        size_t kvoff;
        if (e.kv_mode == 0) kvoff = ((size_t)e.rows.user[row] * e.H * e.Pmax + pos) * e.dh;
        else kvoff = (size_t)e.rows.slot[row] * e.d;
        const size_t hstride = e.kv_mode == 0 ? (size_t)e.Pmax * e.dh : (size_t)e.dh;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = col0 + j * 32 + fr;
          if (col >= N) continue;
          const int which = col / e.d, hc = col - which * e.d;
          const int head = hc / e.dh, ii = hc - head * e.dh;
          float v = acc[i][j][r];
          if (which < 2) {
            const float pv = pb == 1 ? acc[i][j ^ 1][r] : acc[i][j ^ 2][r];
            const int fi = ii & (halfdh - 1);
            const float c = e.cosT[pos * halfdh + fi], s = e.sinT[pos * halfdh + fi];
            v = ii < halfdh ? v * c - pv * s : v * c + pv * s;
          }
          const bf16_t o = f2bf(v);
          if (which == 0) e.q[(size_t)row * e.d + hc] = o;
          else (which == 1 ? e.kdst : e.vdst)[kvoff + head * hstride + ii] = o;
        }
      }
    }
  }
}

// ------------------------------------------------------------------ fp32 path
template <int BMAP>
__global__ void __launch_bounds__(256)
gemm_f32_kernel(const float* __restrict__ A, int lda, const int* __restrict__ Mdev, int N, int K,
                const float* w0, const float* w1, const float* w2, int split, float* __restrict__ C) {
  __shared__ float As[16][65];
  __shared__ float Bs[16][65];
  const int M = *Mdev;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  if (m0 >= M) return;
  const int tid = threadIdx.x, tr = tid / 16, tc = tid % 16;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int i = tid; i < 64 * 16; i += 256) {
      int r = i / 16, k = i % 16;
      int gr = m0 + r < M ? m0 + r : M - 1;
      As[k][r] = A[(size_t)gr * lda + k0 + k];
      int gn = n0 + r < N ? n0 + r : N - 1;
      const float* w;
      if (BMAP == BMAP_PLAIN) w = w0 + (size_t)gn * K;
      else if (BMAP == BMAP_QKV) {
        int which = gn / split;
        w = (which == 0 ? w0 : which == 1 ? w1 : w2) + (size_t)(gn - which * split) * K;
      } else {
        w = (gn < split ? w0 + (size_t)gn * K : w1 + (size_t)(gn - split) * K);
      }
      Bs[k][r] = w[k0 + k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float a[4], bb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[k][tr + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bb[j] = Bs[k][tc + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * bb[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int r = m0 + tr + 16 * i, c = n0 + tc + 16 * j;
      if (r < M && c < N) C[(size_t)r * N + c] = acc[i][j];
    }
}

// Elementwise epilogues of the fp32 path (C is [M, N] fp32).
__global__ void epi_f32_kernel(const float* __restrict__ C, const int* __restrict__ Mdev, int N, int epi,
                               EpiArgs e, int f) {
  const int M = *Mdev;
  const size_t total = (size_t)M * (epi == EPI_GU ? f : N);
  for (size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x; idx < total; idx += (size_t)gridDim.x * blockDim.x) {
    if (epi == EPI_RESID) {
      e.out[idx] += C[idx];
    } else if (epi == EPI_GU) {
      size_t row = idx / f, c = idx % f;
      float g = C[row * N + c], u = C[row * N + f + c];
      reinterpret_cast<float*>(e.hout)[idx] = silu(g) * u;
    } else if (epi == EPI_QKV) {
      int row = (int)(idx / N), col = (int)(idx % N);
      int which = col / e.d, hc = col - which * e.d, head = hc / e.dh, ii = hc - head * e.dh;
      int halfdh = e.dh >> 1, pos = e.rows.pos[row];
      float v = C[idx];
      if (which < 2) {
        int pc = ii < halfdh ? col + halfdh : col - halfdh;
        float pv = C[(size_t)row * N + pc];
        int fi = ii % halfdh;
        float c = e.cosT[pos * halfdh + fi], s = e.sinT[pos * halfdh + fi];
        v = ii < halfdh ? v * c - pv * s : v * c + pv * s;
      }
      if (which == 0) {
        reinterpret_cast<float*>(e.q)[(size_t)row * e.d + hc] = v;
      } else {
        size_t kvoff = e.kv_mode == 0 ? ((size_t)e.rows.user[row] * e.H * e.Pmax + pos) * e.dh
                                      : (size_t)e.rows.slot[row] * e.d;
        size_t hs = e.kv_mode == 0 ? (size_t)e.Pmax * e.dh : (size_t)e.dh;
        reinterpret_cast<float*>(which == 1 ? e.kdst : e.vdst)[kvoff + head * hs + ii] = v;
      }
    } else {
      e.out[idx] = C[idx];
    }
  }
}

// ------------------------------------------------------------------ launchers
using TileBig = Tile<2, 2, 2, 4>;

template <int BMAP, int EPI>
static hipError_t launch_bf16(const GemmCall& g, hipStream_t st) {
  using T = TileBig;
  BArgs b{(const bf16_t*)g.w0, (const bf16_t*)g.w1, (const bf16_t*)g.w2, g.split};
  EpiArgs e{};
  e.out = g.out; e.ldo = g.ldo; e.hout = (bf16_t*)g.hout;
  e.q = (bf16_t*)g.q; e.kdst = (bf16_t*)g.kdst; e.vdst = (bf16_t*)g.vdst;
  e.cosT = g.cosT; e.sinT = g.sinT; e.rows = g.rows; e.kv_mode = g.kv_mode; e.Pmax = g.Pmax;
  e.d = g.d; e.dh = g.dh; e.H = g.H;
  dim3 grid((g.N + T::BN - 1) / T::BN, (g.Mmax + T::BM - 1) / T::BM);
  auto kern = gemm_bf16_kernel<2, 2, 2, 4, BMAP, EPI>;
  static bool attr = false;
  if (!attr) {
    hipError_t err = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, 2 * T::STAGE);
    if (err != hipSuccess) return err;
    attr = true;
  }
  hipLaunchKernelGGL(kern, grid, dim3(T::NT), 2 * T::STAGE, st, (const bf16_t*)g.A, g.lda, g.Mdev, g.N, g.K, b, e);
  return hipGetLastError();
}

hipError_t gemm(const GemmCall& g, hipStream_t st) {
  if (g.bf16) {
    switch (g.kind) {
      case GEMM_QKV: return launch_bf16<BMAP_QKV, EPI_QKV>(g, st);
      case GEMM_GU: return launch_bf16<BMAP_GU, EPI_GU>(g, st);
      case GEMM_RESID: return launch_bf16<BMAP_PLAIN, EPI_RESID>(g, st);
      default: return launch_bf16<BMAP_PLAIN, EPI_STORE>(g, st);
    }
  }
  // fp32: raw product into g.scratch (or straight into the logits), then the
  // elementwise epilogue
  dim3 grid((g.N + 63) / 64, (g.Mmax + 63) / 64);
  const float* A = (const float*)g.A;
  float* C = g.kind == GEMM_STORE ? g.out : g.scratch;
  int bmap = g.kind == GEMM_QKV ? BMAP_QKV : g.kind == GEMM_GU ? BMAP_GU : BMAP_PLAIN;
  if (bmap == BMAP_QKV)
    hipLaunchKernelGGL(gemm_f32_kernel<BMAP_QKV>, grid, dim3(256), 0, st, A, g.lda, g.Mdev, g.N, g.K,
                       (const float*)g.w0, (const float*)g.w1, (const float*)g.w2, g.split, C);
  else if (bmap == BMAP_GU)
    hipLaunchKernelGGL(gemm_f32_kernel<BMAP_GU>, grid, dim3(256), 0, st, A, g.lda, g.Mdev, g.N, g.K,
                       (const float*)g.w0, (const float*)g.w1, nullptr, g.split, C);
  else
    hipLaunchKernelGGL(gemm_f32_kernel<BMAP_PLAIN>, grid, dim3(256), 0, st, A, g.lda, g.Mdev, g.N, g.K,
                       (const float*)g.w0, nullptr, nullptr, g.split, C);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || g.kind == GEMM_STORE) return err;
  EpiArgs e{};
  e.out = g.out; e.ldo = g.ldo; e.hout = (bf16_t*)g.hout;
  e.q = (bf16_t*)g.q; e.kdst = (bf16_t*)g.kdst; e.vdst = (bf16_t*)g.vdst;
  e.cosT = g.cosT; e.sinT = g.sinT; e.rows = g.rows; e.kv_mode = g.kv_mode; e.Pmax = g.Pmax;
  e.d = g.d; e.dh = g.dh; e.H = g.H;
  int epi = g.kind == GEMM_QKV ? EPI_QKV : g.kind == GEMM_GU ? EPI_GU : g.kind == GEMM_RESID ? EPI_RESID : EPI_STORE;
  hipLaunchKernelGGL(epi_f32_kernel, dim3(1024), dim3(256), 0, st, g.scratch, g.Mdev, g.N, epi, e, g.split);
  return hipGetLastError();
}

}  // namespace atspeed
