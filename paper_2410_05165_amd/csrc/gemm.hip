// Dense projections of the decoder block: Y[M, N] = X[M, K] · W[N, K]^T.
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16 (fp32 accumulate), block tile
// BM x BN x 64 fetched by direct global->LDS DMA into two LDS stages
// (XOR-swizzled 16-byte chunks), or three to six for small row counts, wave
// tile TM x TN blocks of 32x32, tile shape chosen by the row count.  Epilogues are
// fused:
//   QKV   rotary embedding on q and k, rounding to bf16, q to its row buffer,
//         k/v scattered into the prefix cache or the tree KV buffer.  The tile's
//         weight rows are interleaved (qkv_logical) so that a column's
//         rotate-half partner is lane ^ 16 of the same MFMA block, one
//         v_permlane16_swap away whatever the tile width;
//   GU    gate and up columns share a tile (first/second half of each wave's
//         blocks), out = bf16(SiLU(gate) * up);
//   RESID residual stream x += acc (fp32); with a partial buffer the k range
//         is split at K/2 into two workgroups per tile, the first adding its
//         product into x and the second storing its own into the buffer (the
//         following RMSNorm adds it), so the o and down projections fill the
//         CUs with 256x256 tiles;
//   STORE fp32 logits.
// M is read from device memory; the grid covers the caller's row count or
// bound (GemmCall::Mmax), and tiles past M exit at once.
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
  float* part;       // RESID split in k: the second half's product [M, ldo] fp32 (null: no split)
  bf16_t* hout;      // GU: [M, f] bf16
  // QKV
  bf16_t* q;         // [M, d]
  bf16_t* kdst;      // prefix cache or tree KV base of this layer
  bf16_t* vdst;
  const float* cosT; // fp32 path: [max_pos, dh/2]
  const float* sinT;
  const float* ropeT; // bf16 path: [max_pos][16][4] (cos, sin), rotary index 16*b + i at [pos][i][b]
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
  static constexpr int A_BYTES = BM * 128;
  static constexpr int B_BYTES = BN * 128;
  static constexpr int STAGE = A_BYTES + B_BYTES;
};

typedef __attribute__((address_space(3))) void lds_void_t;

// LDS swizzle of the 128-byte tile rows: logical 16-byte chunk c of row r sits
// at physical chunk c ^ swz(r).  A fragment read has 16 lanes on 16 consecutive
// rows in one LDS cycle, and a row covers half of the 64 banks, so the 8 even
// rows must use 8 distinct chunks and so must the 8 odd ones: (r >> 1) & 7
// does that (r & 7 would put rows r and r + 8 on the same banks).
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// Column order of the q/k/v product (bf16 path).  Within each head, the 32
// columns of MFMA block b hold rotary indices 16b .. 16b+15 of the head's first
// half in lanes 0..15 and the same indices of its second half in lanes 16..31,
// so every column's rotate-half partner is lane ^ 16 of the same block.  Maps a
// column's place pp within its head (as the tile holds it) to its column in
// the head (d_head 64 or 128); a bijection on 0 .. d_head-1 that keeps runs of
// 16 columns, and so 16-byte chunks of the bf16 output, contiguous.
__device__ __forceinline__ int qkv_logical(int pp, int halfdh) {
  return ((pp >> 5) << 4) + (pp & 15) + ((pp & 16) ? halfdh : 0);
}

// One k-tile (64 columns of A and W) into an LDS stage with direct global->LDS
// DMA (global_load_lds_dwordx4): each wave instruction fills 1 KB = 8 rows of
// 128 B; lane i lands at byte 16*i, i.e. row i/8, physical chunk i%8, and so
// fetches logical chunk (i%8) ^ swz(row) -- the XOR swizzle the fragment reads
// undo.  No VGPRs hold the tile.  Each address is a wave-uniform base plus an
// unsigned 32-bit byte offset per lane, so the instruction takes its scalar-base
// form (one VGPR per address instead of a 64-bit pair: fewer live registers,
// measured 3-7% faster on the 7B projections); the byte offsets stay below 2^32
// (activation and weight buffers are below 2^31 elements).
template <int NA, int NB>
__device__ __forceinline__ void load_stage(unsigned char* stage, int wave, const bf16_t* A, const int* a_off,
                                           const bf16_t* const* Bp, const int* b_off, int k0, int a_bytes) {
#pragma unroll
  for (int j = 0; j < NA; ++j)
    __builtin_amdgcn_global_load_lds((void*)(reinterpret_cast<const unsigned char*>(A) + (uint32_t)(a_off[j] + k0) * 2u),
                                     (lds_void_t*)(stage + (wave * NA + j) * 1024), 16, 0, 0);
#pragma unroll
  for (int j = 0; j < NB; ++j)
    __builtin_amdgcn_global_load_lds(
        (void*)(reinterpret_cast<const unsigned char*>(Bp[j]) + (uint32_t)(b_off[j] + k0) * 2u),
        (lds_void_t*)(stage + a_bytes + (wave * NB + j) * 1024), 16, 0, 0);
}

// The same stage load as untracked inline-asm DMA, for the pipelines with more
// than two stages: the compiler counts only a few LDS-DMA stores in flight and
// would drain all of them once per round, so these loads are issued where it
// does not see them and the pipeline waits with an explicit vmcnt.  The asm
// writes M0 (the LDS address) itself.  M0 is a reserved register, so the
// compiler ignores its clobber (and warns); that is safe because the kernels
// that use these loads contain no M0 use of the compiler's own (the two-stage
// kernels, whose builtin DMA sets M0, contain no such asm).  Binding the
// address to M0 as an asm operand instead was tried and faulted the GPU.
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v), hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}
template <int NA, int NB>
__device__ __forceinline__ void load_stage_u(unsigned char* stage, int wave, const bf16_t* A, const int* a_off,
                                             const bf16_t* const* Bp, const int* b_off, int k0, int a_bytes) {
  const void* Au = uniform_ptr(A);
#pragma unroll
  for (int j = 0; j < NA; ++j) {
    const uint32_t lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_t*)(stage + (wave * NA + j) * 1024));
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"((uint32_t)(a_off[j] + k0) * 2u),
                 "s"(Au) : "memory", "m0");
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const uint32_t lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_t*)(stage + a_bytes + (wave * NB + j) * 1024));
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"((uint32_t)(b_off[j] + k0) * 2u),
                 "s"(uniform_ptr(Bp[j])) : "memory", "m0");
  }
}

// One LDS stage (64 columns of k) through the MFMAs.  Fragments of k-step kk+1
// are read into a second register set while the MFMAs of step kk issue, so the
// LDS latency hides behind matrix work instead of stalling every step.
template <int WM, int WN, int TM, int TN>
__device__ __forceinline__ void mma_stage(const unsigned char* stage, int wave_m, int wave_n, int fr, int fc,
                                          f32x16_t (&acc)[TM][TN], int a_bytes) {
  bf16x8_t af[2][TM], bfr[2][TN];
  auto read = [&](int kk, bf16x8_t (&a)[TM], bf16x8_t (&b)[TN]) {
    const int ch = kk * 2 + fc;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = wave_m * TM * 32 + i * 32 + fr;
      a[i] = *reinterpret_cast<const bf16x8_t*>(stage + r * 128 + ((ch ^ swz(r)) << 4));
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int r = wave_n * TN * 32 + j * 32 + fr;
      b[j] = *reinterpret_cast<const bf16x8_t*>(stage + a_bytes + r * 128 + ((ch ^ swz(r)) << 4));
    }
  };
  read(0, af[0], bfr[0]);
  // the scheduling groups below describe the whole stage in order: these reads,
  // then per k-step an MFMA / next-step-read alternation (mask 0x008 = MFMA,
  // 0x100 = DS read), then the last step's MFMAs
  __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);
  static_for<4>([&](auto KK) {
    constexpr int kk = decltype(KK)::value;
    constexpr int cur = kk & 1, nxt = cur ^ 1;
    if constexpr (kk + 1 < 4) read(kk + 1, af[nxt], bfr[nxt]);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
    if constexpr (kk + 1 < 4) {
      static_for<TM + TN>([&](auto) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      });
      __builtin_amdgcn_sched_group_barrier(0x008, TM * TN - (TM + TN), 0);
    } else {
      __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0);
    }
  });
}

template <int WM, int WN, int TM, int TN, int BMAP, int EPI, int NS>
__global__ void __launch_bounds__(64 * WM * WN)
gemm_bf16_kernel(const bf16_t* __restrict__ A, int lda, const int* __restrict__ Mdev, int Mt, int N, int K,
                 BArgs b, EpiArgs e) {
  using T = Tile<WM, WN, TM, TN>;
  constexpr int NW = WM * WN;
  static_assert(NW == 1 || NW == 2 || NW == 4 || NW == 8, "one, two, four or eight waves");
  static_assert(NS >= 2 && NS <= 8, "two to eight LDS stages");
  constexpr int NA = T::BM / (8 * NW);   // wave instructions per stage for A (8 rows of 128 B each)
  constexpr int NB = T::BN / (8 * NW);
  // two stages: two named arrays (see the pipeline below); more: one array of NS
  __shared__ __align__(1024) unsigned char st0[NS == 2 ? T::STAGE : 16];
  __shared__ __align__(1024) unsigned char st1[NS == 2 ? T::STAGE : 16];
  __shared__ __align__(1024) unsigned char stn[NS > 2 ? NS : 1][NS > 2 ? T::STAGE : 16];
  const int M = *Mdev;
  // XCD-aware tile order: workgroup L is dispatched to XCD L % 8; XCD x owns the
  // contiguous range x*per .. x*per+per-1 of the tiles.  Tiles are numbered in
  // groups of GM M-tiles, N-major inside a group, so the workgroups that run at
  // once on an XCD cover a few M-tiles times a few N-tiles and share both their
  // activation and their weight slices in its L2 (numbering all M-tiles first
  // gives each running workgroup its own activation slice once M is large: at
  // 38,400 rows that fetched 28 GB per gate/up launch).  GM = 4 measured best
  // over 1,920-38,400 rows: with many rows the activations, not the weights,
  // fall out of the Infinity Cache, so an activation slice should serve more
  // N-tiles than a weight slice serves M-tiles.  The last group takes the
  // remainder (GM to 2 GM - 1 M-tiles): a group of one or two M-tiles would
  // spread over all N-tiles and make its XCDs stream the whole weight matrix
  // for a few rows (with five 64-row tiles that cost the 320-row step 4%).
  // A RESID call with e.part splits k in two halves at K/2 for every row count
  // (so a row's arithmetic never depends on the batch): workgroups of the
  // first half add their product into the residual, those of the second store
  // theirs into e.part, and the next row kernel adds the two.
  const int kparts = (EPI == EPI_RESID && e.part != nullptr) ? 2 : 1;
  const int Nt = (N + T::BN - 1) / T::BN;
  const int tiles1 = Mt * Nt, ntiles = tiles1 * kparts, per = (ntiles + 7) >> 3;
  const int L = blockIdx.x;
  const int tk = (L & 7) * per + (L >> 3);
  if (tk >= ntiles) return;
  const int ks = tk / tiles1, t = tk - ks * tiles1;
  const int kbase = ks * (K / kparts);
  constexpr int GM = 4;
  const int ngrp = Mt / GM > 0 ? Mt / GM : 1;                 // the last group takes the remainder
  const int g0 = t / (GM * Nt), grp = g0 < ngrp - 1 ? g0 : ngrp - 1;
  const int gm0 = grp * GM, gsz = grp == ngrp - 1 ? Mt - gm0 : GM;
  const int tr = t - gm0 * Nt;
  const int tile_n = tr / gsz, tile_m = gm0 + tr - tile_n * gsz;
  const int m0 = tile_m * T::BM;
  if (m0 >= M) return;
  // wave index in a scalar register: the DMA row bases and the weight choice
  // derived from it are then wave-uniform
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wave_m = wave / WN, wave_n = wave % WN;
  const int lrow = lane >> 3;

  // per-lane element offsets of the 16-byte chunks this lane fetches
  int a_off[NA], b_off[NB];
#pragma unroll
  for (int j = 0; j < NA; ++j) {
    int r = (wave * NA + j) * 8 + lrow;
    int gr = m0 + r;
    gr = gr < M ? gr : M - 1;
    a_off[j] = gr * lda + kbase + ((lane & 7) ^ swz(r)) * 8;
  }
  // Weight rows of the B tile.  DMA instruction j fills tile rows r0 .. r0+7
  // (r0 = (wave*NB + j)*8), all from one weight matrix Bp[j], chosen from r0
  // alone so that its base stays wave-uniform (d_model and d_ffn are multiples
  // of 8, so no instruction straddles two matrices).
  const bf16_t* Bp[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int r0 = (wave * NB + j) * 8, r = r0 + lrow;
    int row;
    if (BMAP == BMAP_GU) {
      // gate rows in the first half of each wave's blocks, the matching up rows in the second
      constexpr int half = TN / 2;
      const int wn = r / (TN * 32), blk = (r / 32) % TN, cc = r % 32;
      row = tile_n * (T::BN / 2) + wn * (half * 32) + (blk % half) * 32 + cc;
      row = row < b.split ? row : b.split - 1;
      Bp[j] = (r0 / 32) % TN >= half ? b.w1 : b.w0;
    } else if (BMAP == BMAP_QKV) {
      // tile row = column of [q | k | v] (3 d_model), rows past it clamped to the last
      int p = tile_n * T::BN + r;
      p = p < N ? p : N - 1;
      const int p0 = tile_n * T::BN + r0;
      const int which = (p0 < N ? p0 : N - 1) / b.split;
      const int hc = p - which * b.split, pp = hc & (e.dh - 1);
      row = hc - pp + qkv_logical(pp, e.dh >> 1);
      Bp[j] = which == 0 ? b.w0 : (which == 1 ? b.w1 : b.w2);
    } else {
      row = tile_n * T::BN + r;
      row = row < N ? row : N - 1;
      Bp[j] = b.w0;
    }
    b_off[j] = row * K + kbase + ((lane & 7) ^ swz(r)) * 8;
  }

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = K / kparts / T::BK;
  const int fr = lane & 31, fc = lane >> 5;
  // Two-stage pipeline: while the MFMAs consume one LDS stage, the DMA of the
  // next k-tile fills the other.  Each stage is its own LDS array, named at
  // compile time, so the compiler sees that a step's DMA and fragment reads
  // touch different objects and inserts no waits between them.
  // nk is even (each k-range is a multiple of 128, checked on the host)
  if constexpr (NS > 2) {
  // NS-stage pipeline (small row counts, where each k-tile's weights arrive
  // cold from HBM): stage s of round kt0 computes k-tile kt0+s while the DMA of
  // k-tiles up to kt0+s+NS-1 is in flight; at each stage end the wave waits
  // until only the newest NS-2 stages' loads are outstanding, then a bare
  // barrier makes every wave's share of the next stage visible.  Empty asm with
  // a memory clobber on both sides keeps fragment reads and DMA issue from
  // moving across the barrier (the barrier intrinsic does not order memory).
  auto stage = [&](auto S) -> unsigned char* { return stn[decltype(S)::value % NS]; };
  constexpr int NLOADS = NA + NB;                 // DMA instructions per stage per lane
  constexpr int ALLOW = NLOADS * (NS - 2);        // loads that may stay in flight at a stage boundary
  constexpr int WAITCNT = (ALLOW & 0xF) | (((ALLOW >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8);
  constexpr int WAITALL = (0x7 << 4) | (0xF << 8);  // vmcnt(0)
  static_assert(ALLOW < 64, "vmcnt holds 6 bits");
  static_for<NS - 1>([&](auto S) {
    constexpr int s_ = decltype(S)::value;
    if (s_ < nk) load_stage_u<NA, NB>(stage(S), wave, A, a_off, Bp, b_off, s_ * 64, T::A_BYTES);
  });
  asm volatile("" ::: "memory");
  if (NS - 2 < nk) __builtin_amdgcn_s_waitcnt(WAITCNT);
  else __builtin_amdgcn_s_waitcnt(WAITALL);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  for (int kt0 = 0; kt0 < nk; kt0 += NS) {
    static_for<NS>([&](auto S) {
      constexpr int s_ = decltype(S)::value;
      const int kt = kt0 + s_;
      if (kt < nk) {
        if (kt + NS - 1 < nk)
          load_stage_u<NA, NB>(stage(std::integral_constant<int, s_ + NS - 1>{}), wave, A, a_off, Bp, b_off,
                               (kt + NS - 1) * 64, T::A_BYTES);
        __builtin_amdgcn_sched_barrier(0);
        mma_stage<WM, WN, TM, TN>(stage(S), wave_m, wave_n, fr, fc, acc, T::A_BYTES);
        asm volatile("" ::: "memory");
        if (kt + NS - 1 < nk) __builtin_amdgcn_s_waitcnt(WAITCNT);
        else __builtin_amdgcn_s_waitcnt(WAITALL);
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
      }
    });
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  } else {
  load_stage<NA, NB>(st0, wave, A, a_off, Bp, b_off, 0, T::A_BYTES);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // sched_barrier(0) after each DMA issue: left free, the scheduler sinks the
  // DMA below the stage's MFMAs, right before the wait that ends the stage,
  // and the load latency is exposed instead of hidden
  for (int kt = 0; kt < nk; kt += 2) {
    load_stage<NA, NB>(st1, wave, A, a_off, Bp, b_off, (kt + 1) * 64, T::A_BYTES);
    __builtin_amdgcn_sched_barrier(0);
    mma_stage<WM, WN, TM, TN>(st0, wave_m, wave_n, fr, fc, acc, T::A_BYTES);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kt + 2 < nk) load_stage<NA, NB>(st0, wave, A, a_off, Bp, b_off, (kt + 2) * 64, T::A_BYTES);
    __builtin_amdgcn_sched_barrier(0);
    mma_stage<WM, WN, TM, TN>(st1, wave_m, wave_n, fr, fc, acc, T::A_BYTES);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  }

  // ---- epilogue.  acc[i][j][r] is row (r/4)*8 + (lane/32)*4 + r%4, column lane%32 of block (i, j).
  const int row0 = m0 + wave_m * TM * 32;
  const int col0 = tile_n * T::BN + wave_n * TN * 32;
  if constexpr (EPI == EPI_STORE || EPI == EPI_RESID) {
    // Branch-free: the accesses go through a buffer resource spanning this
    // tile's valid rows, so the hardware drops stores past it (rows >= M, and
    // columns >= N, which get an out-of-range offset) and returns 0 for such
    // loads.  Guarding each access with a branch instead makes the compiler
    // wait for every store before the next one.  RESID loads all TN x 16
    // residual values of a 32-row block before it adds and stores them.
    const int mrows = M - m0 < T::BM ? M - m0 : T::BM;
    const bool add_old = EPI == EPI_RESID && ks == 0;   // the k-split's second half stores its product alone
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (ks == 0 ? e.out : e.part) + (size_t)m0 * e.ldo, 0, mrows * e.ldo * (int)sizeof(float), 0x00020000);
    const int lrow0 = wave_m * TM * 32;
    // byte offset = row part + column part; a column >= N gets a 1 GiB column
    // part, past the range of any tile's rows
    int coff[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = col0 + j * 32 + fr;
      coff[j] = col < N ? col * (int)sizeof(float) : (1 << 30);
    }
    static_for<TM>([&](auto I) {
      constexpr int i = decltype(I)::value;
      int roff[16];
      static_for<16>([&](auto R) {
        constexpr int r = decltype(R)::value;
        roff[r] = (lrow0 + i * 32 + (r >> 2) * 8 + fc * 4 + (r & 3)) * e.ldo * (int)sizeof(float);
      });
      // residual values loaded for half a 32-row block at a time, all issued
      // before any is used
      static_for<2>([&](auto Hh) {
        constexpr int h0 = decltype(Hh)::value * 8;
        float old[TN][8];
        if (add_old) {
          static_for<8>([&](auto R) {
            constexpr int r = decltype(R)::value;
#pragma unroll
            for (int j = 0; j < TN; ++j)
              old[j][r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, roff[h0 + r] + coff[j], 0, 0));
          });
        }
        static_for<8>([&](auto R) {
          constexpr int r = decltype(R)::value;
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const float v = add_old ? old[j][r] + acc[i][j][h0 + r] : acc[i][j][h0 + r];
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), rs, roff[h0 + r] + coff[j], 0, 0);
          }
        });
      });
    });
  } else {
    // Results are rounded to bf16 into an LDS copy of the output tile (the stage
    // buffers are free now), then written out in 16-byte chunks along rows.
    constexpr int OUTC = EPI == EPI_GU ? T::BN / 2 : T::BN;  // output columns of the tile
    constexpr int OROW = OUTC * 2;                            // bytes per LDS row
    // The whole output tile in the first stage buffer when it fits; otherwise
    // its first half of rows there and the second in the next one.
    constexpr bool ONEBUF = T::BM * OROW <= T::STAGE;
    constexpr int HROWS = ONEBUF ? T::BM : T::BM / 2;
    constexpr int WMH = ONEBUF ? WM : WM / 2;       // wave rows per buffer
    static_assert(ONEBUF || (HROWS * OROW <= T::STAGE && WM % 2 == 0), "each half of the output tile fits a stage");
    unsigned char* const ob0 = NS == 2 ? st0 : stn[0];
    unsigned char* const ob1 = NS == 2 ? st1 : stn[NS > 2 ? 1 : 0];
    bf16_t* ob = reinterpret_cast<bf16_t*>(wave_m < WMH ? ob0 : ob1);
    const int hrow0 = (wave_m % WMH) * TM * 32;
    if constexpr (EPI == EPI_GU) {
      constexpr int half = TN / 2;
      static_for<TM>([&](auto I) {
        constexpr int i = decltype(I)::value;
        static_for<16>([&](auto R) {
          constexpr int r = decltype(R)::value;
          const int hr = hrow0 + i * 32 + (r >> 2) * 8 + fc * 4 + (r & 3);  // row within this half
#pragma unroll
          for (int j = 0; j < half; ++j) {
            const int lc = wave_n * (half * 32) + j * 32 + fr;
            ob[hr * OUTC + lc] = f2bf(silu(acc[i][j][r]) * acc[i][j + half][r]);
          }
        });
      });
    } else {  // EPI_QKV: rotary embedding on q and k (column order of qkv_logical)
      // per block (wave-uniform; d_model and d_head are multiples of 32): which of
      // q, k, v it lies in, and b, its rotary indices being 16b + lane % 16
      int bsel[TN];
      bool rotj[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        int pc = col0 + j * 32;
        pc = pc < N ? pc : N - 32;
        const int wj = pc / e.d;
        rotj[j] = wj < 2;
        bsel[j] = ((pc - wj * e.d) & (e.dh - 1)) >> 5;
      }
      const bool lo = fr < 16;            // first half of the head: x1 cos - x2 sin, else x2 cos + x1 sin
      const int i16 = fr & 15;
      static_for<TM>([&](auto I) {
        constexpr int i = decltype(I)::value;
        // rows in groups of 4: positions, then the (cos, sin) pairs of the group's
        // rows and blocks, all issued before any is used; v columns take cos 1,
        // sin 0 without a branch
        static_for<4>([&](auto Q) {
          constexpr int qg = decltype(Q)::value;
          int pos[4];
          static_for<4>([&](auto R) {
            constexpr int r = decltype(R)::value;
            const int hr = hrow0 + i * 32 + qg * 8 + fc * 4 + r;
            const int row = m0 + (wave_m < WMH ? 0 : HROWS) + hr;
            pos[r] = e.rows.pos[row < M ? row : M - 1];
          });
          // (cos, sin) of each row and block: the block's rotary index picks the
          // pair within the row's table entry by address, so no select on values
          f32x2_t cs[4][TN];
          static_for<4>([&](auto R) {
            constexpr int r = decltype(R)::value;
            const float* t = e.ropeT + ((size_t)pos[r] * 16 + i16) * 8;
#pragma unroll
            for (int j = 0; j < TN; ++j) cs[r][j] = *reinterpret_cast<const f32x2_t*>(t + bsel[j] * 2);
          });
          static_for<4>([&](auto R) {
            constexpr int r = decltype(R)::value;
            constexpr int ra = qg * 4 + r;     // accumulator register of this row
            const int hr = hrow0 + i * 32 + qg * 8 + fc * 4 + r;
            static_for<TN>([&](auto J) {
              constexpr int j = decltype(J)::value;
              const float v = acc[i][j][ra];
              // partner = lane ^ 16: v_permlane16_swap of two copies exchanges
              // the odd 16-lane rows of the first with the even rows of the
              // second, so the first holds the partner in lanes 16..31 and the
              // second in lanes 0..15 (a VALU op, no LDS round trip)
              const auto sw = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
              const float pv = __uint_as_float(lo ? sw[1] : sw[0]);
              const float cb = cs[r][j][0], sb = cs[r][j][1];
              const float c = rotj[j] ? cb : 1.f, sn = rotj[j] ? sb : 0.f;
              // explicit fma of a rounded product: the same arithmetic in every
              // tile shape (free contraction may differ between instantiations,
              // and rows must not depend on the shape their batch got)
              const float ps = pv * sn;
              ob[hr * OUTC + wave_n * TN * 32 + j * 32 + fr] = f2bf(__builtin_fmaf(v, c, lo ? -ps : ps));
            });
          });
        });
      });
    }
    __syncthreads();
    constexpr int CPRW = OUTC / 8;  // 16-byte chunks per output row
    for (int c = tid; c < T::BM * CPRW; c += T::NT) {
      const int lr = c / CPRW, cc = (c % CPRW) * 8;
      const int row = m0 + lr;
      if (row >= M) continue;
      const unsigned char* src = (lr < HROWS ? ob0 : ob1) + (lr % HROWS) * OROW + cc * 2;
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(src);
      if constexpr (EPI == EPI_GU) {
        const int fcol = tile_n * (T::BN / 2) + cc;
        if (fcol < b.split) *reinterpret_cast<u32x4_t*>(e.hout + (size_t)row * b.split + fcol) = v;
      } else {
        const int col = tile_n * T::BN + cc;   // 8 columns of the tile's order, one run of qkv_logical
        if (col >= N) continue;
        const int which = col / e.d, pc = col - which * e.d, pp = pc & (e.dh - 1);
        const int hc = pc - pp + qkv_logical(pp, e.dh >> 1);
        if (which == 0) {
          *reinterpret_cast<u32x4_t*>(e.q + (size_t)row * e.d + hc) = v;
        } else {
          const int head = hc / e.dh, ii = hc - head * e.dh;
          size_t off;
          if (e.kv_mode == 0) off = (((size_t)e.rows.user[row] * e.H + head) * e.Pmax + e.rows.pos[row]) * e.dh + ii;
          else off = (size_t)e.rows.slot[row] * e.d + hc;
          *reinterpret_cast<u32x4_t*>((which == 1 ? e.kdst : e.vdst) + off) = v;
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
// Launch of one instantiation over the tiles of a call.  The widest tiles,
// 256x256 of 8 waves (64x128 each, two waves per SIMD), let one wave's LDS and
// barrier waits hide behind the other's MFMAs.
template <int BMAP, int EPI, int WMW, int WNW, int TMW, int TNW, int NS = 2>
static hipError_t launch_bf16(const GemmCall& g, hipStream_t st) {
  using T = Tile<WMW, WNW, TMW, TNW>;
  BArgs b{(const bf16_t*)g.w0, (const bf16_t*)g.w1, (const bf16_t*)g.w2, g.split};
  EpiArgs e{};
  e.out = g.out; e.ldo = g.ldo; e.hout = (bf16_t*)g.hout;
  e.part = EPI == EPI_RESID ? g.part : nullptr;
  e.q = (bf16_t*)g.q; e.kdst = (bf16_t*)g.kdst; e.vdst = (bf16_t*)g.vdst;
  e.cosT = g.cosT; e.sinT = g.sinT; e.ropeT = g.ropeT; e.rows = g.rows; e.kv_mode = g.kv_mode; e.Pmax = g.Pmax;
  e.d = g.d; e.dh = g.dh; e.H = g.H;
  const int kparts = e.part ? 2 : 1;
  // each k-range is an even number of k-tiles of 64 (two stages)
  if (g.K % (kparts * 128) != 0) return hipErrorInvalidValue;
  const int Mt = (g.Mmax + T::BM - 1) / T::BM, Nt = (g.N + T::BN - 1) / T::BN;
  const int per = (kparts * Mt * Nt + 7) / 8;
  dim3 grid(8 * per);
  auto kern = gemm_bf16_kernel<WMW, WNW, TMW, TNW, BMAP, EPI, NS>;
  hipLaunchKernelGGL(kern, grid, dim3(T::NT), 0, st, (const bf16_t*)g.A, g.lda, g.Mdev, Mt, g.N, g.K, b, e);
  return hipGetLastError();
}

// Tile shape by row count.  A shape's cost is modelled as the number of rounds
// of its tiles over the CUs (256 x the workgroups of that shape one CU holds)
// times the time of one round, t0 + t4k x (k per workgroup) / 4096, fitted to
// measurements on MI355X at the 7B projections for 320 to 4,096 rows: few rows
// leave a 256-row tile mostly empty and give too few tiles to fill the CUs,
// many rows favour the large tiles' higher MFMA rate, and in between the
// better shape is the one whose last round is fuller.  A last round with a
// fraction φ of its slots used costs (partial + (1 - partial) φ) of a round:
// its tiles share the CUs and memory with fewer others (the row shapes were
// fitted with partial 0.5, q/k/v and gate/up with 1).  The shape does not
// change any element's k-order, so results do not depend on it.  g.Mmax is
// the row count of the call when the caller knows it, else an upper bound.
namespace {
constexpr int kCUs = 256;
struct Shape { int bm, bn, per_cu; float t0, t4k; };
// q/k/v: 256x256 (8 waves), 128x256 (8 waves), 64x256 (2 waves, two per CU),
// 256x192 (8 waves; 3 d_model is a multiple of 192, so no ragged column tile);
// (fitted warm); gate/up: the first three, fitted with the weights arriving cold
// from HBM as they do in a forward (picks the fastest measured shape at every
// one of 13 row counts from 320 to 4,096)
// and 64x256 of 8 waves with three stages (one per CU).  The 128x256 and
// 64x256 tiles of 8 waves run three LDS stages (144 and 120 KB), which hides
// the cold weight fetch at a few hundred rows: q/k/v at 320 rows 86 -> 59 us,
// 128x256 q/k/v at 400-640 rows 85-90 -> 70-78 us and gate/up 143-152 ->
// 120-135 us, with cold weights.  The q/k/v constants are scaled from those
// measurements (256x192 keeps 960 rows and more); gate/up keeps its two-stage
// constant, with which the 128x256 tile is picked only where it was already
// fastest (about 640 rows: 152 -> 135 us)
constexpr Shape kQkvShapes[] = {
    {256, 256, 1, 0.f, 98.f}, {128, 256, 1, 0.f, 57.f}, {64, 256, 2, 0.f, 73.f}, {256, 192, 1, 0.f, 83.f},
    {64, 256, 1, 0.f, 46.f}};
constexpr Shape kGuShapes[] = {{256, 256, 1, 0.f, 104.f}, {128, 256, 1, 0.f, 70.f}, {64, 256, 2, 0.f, 78.f}};
// o, down, output head: 256x256, 256x128 (8 waves), 128x128 (4 waves, two per
// CU), 64x64 (2 waves, four per CU)
// (fitted with the weights arriving cold from HBM: within 3% of the fastest
// measured shape at all 12 row counts from 320 to 4,096, for o and for down)
constexpr Shape kRowShapes[] = {
    {256, 256, 1, 25.f, 97.5f}, {256, 128, 1, 10.5f, 70.f}, {128, 128, 2, 14.f, 59.f}, {64, 64, 4, 6.f, 50.f}};
// residual projections also: 128x128 of 4 waves with three stages (one per CU;
// 320 rows: o 33 -> 26 us, down 72 -> 56 us with cold weights; constants from
// those two measurements)
constexpr Shape kResidShapes[] = {
    {256, 256, 1, 25.f, 97.5f}, {256, 128, 1, 10.5f, 70.f}, {128, 128, 2, 14.f, 59.f}, {64, 64, 4, 6.f, 50.f},
    {128, 128, 1, 4.4f, 36.f}};

// Few rows (a decode level of a few users, the verify tree of one user): the
// weight stream is the whole cost, and the tiles above leave most CUs idle (a
// 256-column tile gives q/k/v 48 workgroups).  Narrow tiles with four to six
// LDS stages give 190-380 workgroups, each streaming a thin weight slice.
// Measured at the 7B projections (1-256 rows, cold weights, warm clocks), with
// the time of the cost model's shape in parentheses:
//   1-32 rows    q/k/v 32x64 of two waves (six stages) 26-28 us (54); gate/up
//                64x64 of two waves (four) 42-43 (60-64); o and down 64x32 of
//                two waves (six) 15 and 30 (22 and 50);
//   33-64        q/k/v 64x64 of 2x2 waves of 32x32 (four) 28-31 (two waves of
//                32x64: 32-34); gate/up 64x128 of 2x2 waves (four) 44-45; o and
//                down as above;
//   65-128       one M-tile of 128 rows over four waves instead of two 64-row
//                tiles: q/k/v 128x64 of 2x2 waves 34-38 (38-44), gate/up
//                128x128 of 2x2 waves 48-53 (55-61), o and down 128x32 of four
//                waves in a column 17-18 and 35-39 (17-18 and 36-42), all four
//                stages.
constexpr int kFewRowsQkv = 128, kFewRowsGu = 128, kFewRowsResid = 128, kNarrowRows = 64;
// A little above that (a prompt of one user, the verify tree of a few): one
// M-tile of 192 rows over all the rows, split among four waves so that every
// SIMD of a CU issues MFMAs (the two-wave tiles of the same height leave half
// of them idle), and each weight slice crosses the chip once.  Measured at the
// 7B projections with cold weights, 129-192 rows: q/k/v 192x64 of 2x2 waves
// (four stages) 45-49 instead of 55-60 us, gate/up 192x128 of 2x2 waves (four
// stages, the whole 160 KB of LDS) 55-59 instead of 65-69, o and down 256x32
// of four waves in a column (four stages) 23-24 and 49-54 instead of 24-25
// and 52-55; at 193-256 rows q/k/v 256x64 of 4x2 waves (three stages) 51-54
// instead of 57-60 and o/down 192x64 of 2x2 waves (four stages) 54-56 instead
// of 56-61 us for down.  Above 256 rows the shapes below are as fast or faster.
constexpr int kMidRows = 192, kMidRows2 = 256;
constexpr int kHeadFewRows = 320;

template <int NSH>
int pick_shape(const Shape (&sh)[NSH], int M, int N, int K, int kparts, float partial) {
  int best = 0;
  float best_cost = 0.f;
  for (int i = 0; i < NSH; ++i) {
    const long tiles = kparts * (long)((M + sh[i].bm - 1) / sh[i].bm) * ((N + sh[i].bn - 1) / sh[i].bn);
    const long slots = (long)kCUs * sh[i].per_cu;
    const long full = tiles / slots, rest = tiles - full * slots;
    const float rounds = (float)full + (rest ? partial + (1.f - partial) * (float)rest / (float)slots : 0.f);
    const float cost = rounds * (sh[i].t0 + sh[i].t4k * (float)K / kparts / 4096.f);
    if (i == 0 || cost < best_cost) { best = i; best_cost = cost; }
  }
  return best;
}
}  // namespace

hipError_t gemm(const GemmCall& g, hipStream_t st) {
  if (g.bf16) {
    const int M = g.Mmax > 0 ? g.Mmax : 1;
    switch (g.kind) {
      case GEMM_QKV:
        if (M <= 32) return launch_bf16<BMAP_QKV, EPI_QKV, 1, 2, 1, 1, 6>(g, st);
        if (M <= kNarrowRows) return launch_bf16<BMAP_QKV, EPI_QKV, 2, 2, 1, 1, 4>(g, st);
        if (M <= kFewRowsQkv) return launch_bf16<BMAP_QKV, EPI_QKV, 2, 2, 2, 1, 4>(g, st);
        if (M <= kMidRows) return launch_bf16<BMAP_QKV, EPI_QKV, 2, 2, 3, 1, 4>(g, st);
        if (M <= kMidRows2) return launch_bf16<BMAP_QKV, EPI_QKV, 4, 2, 2, 1, 3>(g, st);
        switch (pick_shape(kQkvShapes, M, g.N, g.K, 1, 1.f)) {
          case 0: return launch_bf16<BMAP_QKV, EPI_QKV, 4, 2, 2, 4>(g, st);
          case 1: return launch_bf16<BMAP_QKV, EPI_QKV, 4, 2, 1, 4, 3>(g, st);
          case 2: return launch_bf16<BMAP_QKV, EPI_QKV, 1, 2, 2, 4>(g, st);
          case 3: return launch_bf16<BMAP_QKV, EPI_QKV, 4, 2, 2, 3>(g, st);
          default: return launch_bf16<BMAP_QKV, EPI_QKV, 2, 4, 1, 2, 3>(g, st);
        }
      case GEMM_GU:
        if (M <= 32) return launch_bf16<BMAP_GU, EPI_GU, 2, 1, 1, 2, 4>(g, st);
        if (M <= kNarrowRows) return launch_bf16<BMAP_GU, EPI_GU, 2, 2, 1, 2, 4>(g, st);
        if (M <= kFewRowsGu) return launch_bf16<BMAP_GU, EPI_GU, 2, 2, 2, 2, 4>(g, st);
        if (M <= kMidRows) return launch_bf16<BMAP_GU, EPI_GU, 2, 2, 3, 2, 4>(g, st);
        switch (pick_shape(kGuShapes, M, g.N, g.K, 1, 1.f)) {
          case 0: return launch_bf16<BMAP_GU, EPI_GU, 4, 2, 2, 4>(g, st);
          case 1: return launch_bf16<BMAP_GU, EPI_GU, 4, 2, 1, 4, 3>(g, st);
          default: return launch_bf16<BMAP_GU, EPI_GU, 1, 2, 2, 4>(g, st);
        }
      case GEMM_RESID:
        if (M <= kNarrowRows) return launch_bf16<BMAP_PLAIN, EPI_RESID, 2, 1, 1, 1, 6>(g, st);
        if (M <= kFewRowsResid) return launch_bf16<BMAP_PLAIN, EPI_RESID, 4, 1, 1, 1, 4>(g, st);
        if (M <= kMidRows) return launch_bf16<BMAP_PLAIN, EPI_RESID, 4, 1, 2, 1, 4>(g, st);
        if (M <= kMidRows2) return launch_bf16<BMAP_PLAIN, EPI_RESID, 2, 2, 3, 1, 4>(g, st);
        switch (pick_shape(kResidShapes, M, g.N, g.K, g.part ? 2 : 1, 0.5f)) {
          case 0: return launch_bf16<BMAP_PLAIN, EPI_RESID, 4, 2, 2, 4>(g, st);
          case 1: return launch_bf16<BMAP_PLAIN, EPI_RESID, 4, 2, 2, 2>(g, st);
          case 2: return launch_bf16<BMAP_PLAIN, EPI_RESID, 2, 2, 2, 2>(g, st);
          case 3: return launch_bf16<BMAP_PLAIN, EPI_RESID, 1, 2, 2, 1>(g, st);
          default: return launch_bf16<BMAP_PLAIN, EPI_RESID, 2, 2, 2, 2, 3>(g, st);
        }
      default:
        // the item rows of the output head (1,024 columns): up to a few hundred
        // rows 64x32 tiles of two waves with six stages give twice the
        // workgroups of the model's pick and stream the head in 20-22 instead of
        // 32-37 us (1-320 rows, warm clocks)
        if (M <= kHeadFewRows) return launch_bf16<BMAP_PLAIN, EPI_STORE, 2, 1, 1, 1, 6>(g, st);
        switch (pick_shape(kRowShapes, M, g.N, g.K, 1, 0.5f)) {
          case 0: return launch_bf16<BMAP_PLAIN, EPI_STORE, 4, 2, 2, 4>(g, st);
          case 1: return launch_bf16<BMAP_PLAIN, EPI_STORE, 4, 2, 2, 2>(g, st);
          case 2: return launch_bf16<BMAP_PLAIN, EPI_STORE, 2, 2, 2, 2>(g, st);
          default: return launch_bf16<BMAP_PLAIN, EPI_STORE, 1, 2, 2, 1>(g, st);
        }
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
