// LM-head forward (logits + vocab-chunked online log-sum-exp + sampled-token gather),
// the GRPO/DAPO/GSPO loss coefficient, and the LM-head backward, for gfx950.
//
// Sec. 3.2 (post-pruning evaluation) and Sec. 3.1 (Eq. 1, Eq. grad).  With P the softmax
// of z = H W^T and g = dL/dlogp:  dZ = g (onehot(y) - P),  dH = dZ W,  dW = dZ^T H.
//
// One tiled GEMM kernel does the three contractions.  C[m, n] = sum_k A[m, k] B[n, k]
// with 256 x 256 block tiles and LDS double buffering:
//   bf16: 8 wavefronts of 128 x 64, v_mfma_f32_16x16x32_bf16, 64-wide K steps, operands moved
//         by direct global->LDS loads;
//   f32:  4 wavefronts of 128 x 128, v_mfma_f32_32x32x2_f32, register-staged loads.
// Work is cut into slabs of whole sequences; per slab:
//   FWD  C = W . H_slab^T  (rows = vocab, cols = tokens, K = d).  Epilogue: per token,
//        the block's max and sum exp(z - s_t) over its 256 vocab rows (in-lane over 32
//        values, two lane-row swaps, one LDS exchange), the sampled token's logit, and
//        E1[t][v] = exp(z - s_t) (s_t = 0 unless exp(z) would leave float range).
//   merge   partials -> lse, logp, row max; rows whose max is too far from s_t get
//           s_t = max_t and their token block is evaluated again (rare), then merge again.
//   loss    g_t and c_t = g_t exp(s_t - lse_t) per token (one block per sequence).  With a
//           backward it also folds the one-hot term into the exp-logits: since
//           g_t = c_t exp(lse_t - s_t), E1[t][y_t] -= exp(lse_t - s_t) makes
//           c_t E1[t][v] = g_t (P[t][v] - [v = y_t]) = -dZ[t][v] for every v.
//   DH   C = E1 . W^T  (rows = tokens, cols = d, K = vocab):  dH[t] = -c_t C[t].
//   DW   with Bd[n][t] = c_t H[t][n] (K = tokens; E1 is read K-major through transposing LDS
//        reads): bf16 computes C' = Bd . E1 (rows = d, cols = vocab), f32 computes
//        C = E1^T . Bd^T (rows = vocab, cols = d):  dW[v] (+)= -C[v].
// Nothing of size [T, V] exists: the exp-logit buffer holds one slab, [slab, V], and the
// default slab (32768 tokens) does not grow with T.
#include <algorithm>
#include <cstdlib>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace fastrl {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBM = 256, kBN = 256;

// MODE_DWT: the bf16 dW GEMM computed transposed, dW^T = Bd E (rows = hidden columns, cols =
// vocab rows, K = tokens), so that it runs on the 8-wavefront engine with E as a K-major B
enum GemmMode { MODE_FWD = 0, MODE_DH = 1, MODE_DW = 2, MODE_DWT = 3 };

// wavefront geometry of the 256 x 256 block tile: every bf16 GEMM runs 8 wavefronts (two per
// SIMD) of 128 x 64 on 16 x 16 x 32 MFMAs; every float32 GEMM runs 4 wavefronts of 128 x 128
// on 32 x 32 MFMAs
template <typename T, int MODE>
struct Geo {
  static constexpr bool W8 = sizeof(T) == 2;
  static_assert(MODE != (W8 ? MODE_DW : MODE_DWT), "dW runs transposed in bf16 only");
  static constexpr int THREADS = W8 ? 512 : 256, WAVES_N = W8 ? 4 : 2, NI = W8 ? 2 : 4,
                       WPE = W8 ? 2 : 1;
};

template <typename T>
struct Eng;

template <>
struct Eng<uint16_t> {     // bfloat16 operands
  static constexpr int BK = 64;
  static constexpr int KP = 8;             // row padding (elements) against bank conflicts
  static constexpr int LD = BK + KP;       // LDS row stride in elements
  static constexpr int VEC = 8;            // elements per 16-byte vector
  static constexpr int KSTEP = 16;         // K per MFMA
};
template <>
struct Eng<float> {        // float32 operands
  static constexpr int BK = 16;
  static constexpr int KP = 4;
  static constexpr int LD = BK + KP;
  static constexpr int VEC = 4;
  static constexpr int KSTEP = 2;
};

struct GemmParams {
  const void* A;            // [M, lda]
  int64_t lda;
  int32_t M;
  const void* B;            // [N rows, ldb] (rows via b_rows when non-null)
  int64_t ldb;
  int32_t N;
  const int32_t* b_rows;    // FWD: row_index (nullable) offset to the slab
  int64_t b_row_base;       // FWD: first kept token of the slab
  int32_t K;
  int32_t nmb, nnb;         // block grid (M blocks, N blocks)
  int32_t group;            // tile order: M-blocks per sweep over the N-blocks (tile_group)
  // ---- FWD epilogue
  float* pmax;              // [nmb][ldp]
  float* psum;              // [nmb][ldp]
  float* psz;               // [nmb][ldp] or NULL: sum of exp(z - ref) * z (entropy)
  int64_t ldp;
  float* zlab;              // [slab]
  const int32_t* yslab;     // [slab] label of each slab token (-1: invalid)
  const float* shift;       // [slab] s_t (nullable = 0)
  void* E1;                 // [slab rows][ldE1 = V_pad]   E1[t][v] = exp(z[t][v] - s_t)
  int64_t ldE1;
  int32_t Vreal;
  int32_t store_e;          // 0: partials only, 1: partials + E, 2: same for redo blocks
  const int32_t* redo_blk;  // [nnb] token blocks to evaluate again (store_e == 2)
  const int32_t* redo_any;  // nonzero iff some token block of the slab is marked
  // ---- DH epilogue
  void* dH;                 // [.., d] at slab offset
  int32_t dH_bf16;
  const float* cslab;       // [slab]
  int32_t d;
  // ---- DW epilogue
  float* dW;                // [V, d]
  int32_t dW_acc;           // add to dW (later slabs) instead of overwriting it
  int32_t* status;
};

// Tile order: consecutive blocks are dealt round-robin to the 8 XCDs and run at about the same
// time, so the order of logical tiles decides which operand strips are in use together.  A group
// of M-blocks shares each sweep over the N-blocks (p.group, chosen per shape on the host by
// tile_group).  Logits GEMM (short K): 32 at d = 3584, so each XCD holds 4 vocab blocks x 8
// token blocks of the 256 tiles in flight and all XCDs read the same 8 hidden row blocks.
// Backward GEMMs (long K): 4 at d = 3584; all XCDs walk neighbouring tiles through K together,
// so a strip that several XCDs read is fetched once into the shared last-level cache (giving
// each XCD its own contiguous range of tiles measured 2-4% slower here).
// spins of a split-barrier wait before it gives up (each spin one LDS read, ~0.1 us; a
// wavefront normally waits for a few hundred cycles at most)
constexpr int kSyncSpins = 1 << 16;
template <int MODE>
__device__ __forceinline__ void tile_coords(int& mb, int& nb, int nmb, int nnb, int b, int group) {
  // the groups are vocab blocks in both dW forms: M blocks of MODE_DW, N blocks of MODE_DWT
  constexpr bool GN = MODE == MODE_DWT;
  const int ng = GN ? nnb : nmb, ns = GN ? nmb : nnb;
  const int per_group = group * ns;
  const int gid = b / per_group;
  const int first = gid * group;
  const int gsz = min(ng - first, group);
  const int in = b % per_group;
  const int a = first + in % gsz, sweep = in / gsz;
  mb = GN ? sweep : a;
  nb = GN ? a : sweep;
}

template <typename T>
__device__ __forceinline__ void load_vec(const T* p, bool ok, u32x4_t& v) {
  if (ok) v = *reinterpret_cast<const u32x4_t*>(p);
  else v = u32x4_t{0u, 0u, 0u, 0u};
}

template <typename T>
__device__ __forceinline__ float to_f32(T x);
template <>
__device__ __forceinline__ float to_f32<uint16_t>(uint16_t x) { return bf16_to_f32(x); }
template <>
__device__ __forceinline__ float to_f32<float>(float x) { return x; }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ uint16_t from_f32<uint16_t>(float x) { return f32_to_bf16(x); }
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }

// accumulator (mi, ni, r) -> (row, col) inside the 256 x 256 block tile
__device__ __forceinline__ int acc_row(int wm, int mi, int r, int lane) {
  return wm * 128 + mi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
}
template <typename T, int MODE>
__device__ __forceinline__ int acc_col(int wn, int ni, int lane) {
  return wn * (kBN / Geo<T, MODE>::WAVES_N) + ni * 32 + (lane & 31);
}

typedef __attribute__((address_space(3))) void lds_void_t;

// bf16 main loop of the logits GEMM (z = W h: A = LM-head rows, B = gathered hidden rows, K = d),
// the dhidden GEMM (A = the slab's exp-logit rows, B = W^T rows, K = padded vocab) and the
// transposed dW GEMM (A = Bd rows, B = the exp-logit tile read K-major, K = padded slab).
// Eight wavefronts (two per SIMD, so one can issue MFMAs while the other waits on memory) each
// own a 128 x 64 part of the block tile.  LDS holds two stages of a 256 x 64 A tile and a
// 256 x 64 B tile (32 KB each), written by direct global->LDS loads (global_load_lds_dwordx4):
// one load instruction moves 1 KB, lane l writing its 16-byte slot l; each wavefront moves
// 4 KB of each operand per tile.  Tile kt+1 is in flight while tile kt is multiplied;
// fragments of k-step kk+1 are read while the MFMAs of k-step kk run.  The MFMAs are
// v_mfma_f32_16x16x32_bf16 (8 x 4 tiles of 16 x 16 per wavefront, two 32-k steps per tile):
// per FLOP they move less accumulator data through the register file than 32 x 32 x 16, and
// measured 7% faster on the logits GEMM and 4% on dhidden (where this engine also beat a
// four-wavefront one, as it does on dW); lane l holds rows 4 (l / 16) .. 4 (l / 16) + 3 of
// column l % 16 of each 16 x 16 tile.
//
// LDS layout (rows of 64 k = 128 B): row r keeps its k-chunk c (8 bf16) in slot
// c ^ ((r >> 1) & 7).  The LDS serves a 16-byte-per-lane read 16 lanes (256 B, 64 banks) at a
// time, and rows r..r+15 of a fragment then land on 16 distinct 16-byte bank groups; the
// swizzle is applied on the global side (each lane loads the chunk that belongs in its slot).
template <int MODE>
__device__ __forceinline__ void mainloop_bf16_dma(const GemmParams& p, int m0, int n0,
                                                  f32x4_t (&acc)[8][4], uint16_t* smem) {
  constexpr int BK = 64;
  constexpr int TILE = kBM * BK;  // elements per operand per stage
  constexpr bool BKM = MODE == MODE_DWT;  // B stored K-major (B[n][k] at k * ldb + n)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const uint16_t* Ag = static_cast<const uint16_t*>(p.A);
  const uint16_t* Bg = static_cast<const uint16_t*>(p.B);
  const int lrow = lane >> 3;
  // global k-chunk this lane moves into its slot; rows r = 32 wave + 8 j + lrow, so
  // ((r >> 1) & 7) = 4 (j & 1) + (lrow >> 1)
  const int gch[2] = {(lane & 7) ^ (lrow >> 1), (lane & 7) ^ (4 | (lrow >> 1))};
  int64_t arow[4], brow[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = wave * 32 + j * 8 + lrow;
    const int ra = min(m0 + r, p.M - 1);  // rows past the edge load a valid row; their
    arow[j] = int64_t(ra) * p.lda;        // results are never stored
    if constexpr (BKM) {
      // K-major B tile: 64 k-rows of 256 n (512 B); load j of this wavefront fills k-rows
      // 8 wave + 2 j and the next, lane l slot l % 32 of row 8 wave + 2 j + l / 32, with the
      // n-chunk that belongs there (slot = chunk ^ kmaj_swz(k))
      const int k = wave * 8 + 2 * j + (lane >> 5);
      const int swz = ((k & 3) << 1) | (((k >> 3) & 1) << 3);
      brow[j] = int64_t(k) * p.ldb + n0 + (((lane & 31) ^ swz) << 3);
    }
  }
  if constexpr (!BKM) {
    // B rows, gathered through b_rows when given: the four index loads are issued together
    // (one memory round trip before the first tile load, not four one after the other)
    int64_t bi[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) bi[j] = min(n0 + wave * 32 + j * 8 + lrow, p.N - 1) + p.b_row_base;
    if (p.b_rows) {
      int32_t g[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) g[j] = __builtin_nontemporal_load(p.b_rows + bi[j]);
#pragma unroll
      for (int j = 0; j < 4; ++j) bi[j] = g[j];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) brow[j] = bi[j] * p.ldb;
  }
  // K-major B fragments (ds_read_b64_tr_b16): in 16-lane group g, lane jj reads 4 n of k-row
  // 8 g + 4 s + jj / 4 (s = first / second 4 k of the lane's 8) at n = 16 j + 4 (jj % 4) of
  // the wavefront's 64 columns, and receives the 4 k of column n = 16 j + jj.  The row swizzle
  // puts the 8 rows that lanes 0-31 (and 32-63) read on 16 distinct 16-byte bank groups.
  int bfo[4];
  if constexpr (BKM) {
    const int g = lane >> 4, jj = lane & 15;
    const int swz = ((jj >> 2) << 1) | ((g & 1) << 3);  // kmaj_swz of the rows this lane reads
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = wn * 64 + 16 * j + 4 * (jj & 3);
      bfo[j] = (8 * g + (jj >> 2)) * kBN + (((n >> 3) ^ swz) << 3) + (n & 7);
    }
  }
  // The transposing reads are issued as inline assembly: before the builtin form the compiler
  // waits for every outstanding direct-to-LDS load (it cannot tell the two stages apart), which
  // drains the next tile's prefetch in every k-step (measured 10% slower).  Their results are
  // waited for explicitly (frag_wait) before the MFMAs that read them, and before the barrier
  // that hands their stage back to the loads.
  uint32_t bfa[4];  // LDS byte addresses of this lane's K-major B fragments in stage 0
  if constexpr (BKM) {
    typedef __attribute__((address_space(3))) const uint16_t lds_u16_t;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      bfa[j] = uint32_t(uintptr_t((lds_u16_t*)(smem + TILE + bfo[j])));
  }
  // the B fragments pass through the wait as operands, so no use of them can precede it
  auto frag_wait = [&](bf16x8_t (&fb)[4]) {
    if constexpr (BKM) {
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(fb[0]), "+v"(fb[1]), "+v"(fb[2]), "+v"(fb[3])
                   :
                   : "memory");
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  const int K = p.K;
  const int nk = (K + BK - 1) / BK;
  const bool ktail = (K % BK) != 0;
  auto issue = [&](int kt, int stage) {
    // clamp the chunk so a partial last tile never reads past the end of a row
    const int kc0 = min(kt * BK + gch[0] * 8, K - 8);
    const int kc1 = min(kt * BK + gch[1] * 8, K - 8);
    uint16_t* sa = smem + stage * 2 * TILE + wave * 32 * BK;
    uint16_t* sb = sa + TILE;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kc = (j & 1) ? kc1 : kc0;
      __builtin_amdgcn_global_load_lds(Ag + arow[j] + kc, (lds_void_t*)(sa + j * 8 * BK), 16, 0, 0);
      // (K-major B: k-rows 8 wave + 2 j, + 1 start at the same LDS offset as rows 32 wave + 8 j)
      const uint16_t* bsrc = BKM ? Bg + brow[j] + int64_t(kt) * BK * p.ldb : Bg + brow[j] + kc;
      __builtin_amdgcn_global_load_lds(bsrc, (lds_void_t*)(sb + j * 8 * BK), 16, 0, 0);
    }
  };
  auto zero_tail = [&](int kt, int stage) {  // this lane's slots past K in tile kt
    uint16_t* sa = smem + stage * 2 * TILE + wave * 32 * BK + lane * 8;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (kt * BK + gch[j & 1] * 8 >= K) {
        *reinterpret_cast<u32x4_t*>(sa + j * 8 * BK) = u32x4_t{0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4_t*>(sa + TILE + j * 8 * BK) = u32x4_t{0u, 0u, 0u, 0u};
      }
    }
  };
  const int sw = ((lane & 15) >> 1) & 7;  // ((row >> 1) & 7) of the fragment rows this lane reads
  // fragments of the 32-k step kk (0, 1): A rows wm*128 + i*16 + (lane & 15) and B rows
  // wn*64 + j*16 + (lane & 15), k-chunk 4 kk + lane / 16 (8 consecutive k per lane)
  auto frags = [&](int stage, int kk, bf16x8_t (&fa)[8], bf16x8_t (&fb)[4]) {
    const uint16_t* as = smem + stage * 2 * TILE;
    const uint16_t* bs = as + TILE;
    const int slot = ((kk * 4 + (lane >> 4)) ^ sw) * 8;
    auto read_a = [&](int i) {
      fa[i] = *reinterpret_cast<const bf16x8_t*>(as + (wm * 128 + i * 16 + (lane & 15)) * BK + slot);
    };
    if constexpr (BKM) {
      // program order A0 B0 A1 B1 .. A3 B3 A4 .. A7: the reads stay in this order, so pinning
      // the A reads among the MFMAs spreads the B reads too
      const uint32_t sofs = uint32_t(stage) * (2 * TILE * 2);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        read_a(j);
        typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
        u32x2_t h0, h1;
        const uint32_t a = bfa[j] + sofs;
        if (kk == 0) {
          asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(h0) : "v"(a) : "memory");
          asm volatile("ds_read_b64_tr_b16 %0, %1 offset:2048" : "=v"(h1) : "v"(a) : "memory");
        } else {
          asm volatile("ds_read_b64_tr_b16 %0, %1 offset:16384" : "=v"(h0) : "v"(a) : "memory");
          asm volatile("ds_read_b64_tr_b16 %0, %1 offset:18432" : "=v"(h1) : "v"(a) : "memory");
        }
        fb[j] = __builtin_bit_cast(bf16x8_t, u32x4_t{h0[0], h0[1], h1[0], h1[1]});
      }
#pragma unroll
      for (int i = 4; i < 8; ++i) read_a(i);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) read_a(i);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        fb[j] = *reinterpret_cast<const bf16x8_t*>(bs + (wn * 64 + j * 16 + (lane & 15)) * BK + slot);
    }
  };
  auto mma = [&](const bf16x8_t (&fa)[8], const bf16x8_t (&fb)[4]) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  };
  auto mma_rows = [&](const bf16x8_t (&fa)[8], const bf16x8_t (&fb)[4], int i0, int i1) {
#pragma unroll
    for (int i = i0; i < i1; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  };
  auto mma_half = [&](const bf16x8_t (&fa)[8], const bf16x8_t (&fb)[4], int h) {
    mma_rows(fa, fb, 4 * h, 4 * h + 4);
  };

  bf16x8_t fa0[8], fb0[4], fa1[8], fb1[4];
  // fragment reads per k-step that the scheduler places: 8 A reads and 4 B reads, or (K-major
  // B) the 8 A reads, each followed in program order by the assembly B reads
  constexpr int NRD = BKM ? 8 : 12;
  // pin the order inside a k-step: the 32 MFMAs of this step with the fragment reads of the
  // next step spread among the first 24 (at most one step's reads in flight, so the wait before
  // the next step's MFMAs is exact, and the last read still has 8 MFMAs to land)
  auto kstep = [&](int stage, int kk_next, bf16x8_t (&fa)[8], bf16x8_t (&fb)[4],
                   bf16x8_t (&na)[8], bf16x8_t (&nb)[4]) {
    frag_wait(fb);
    // raised wave priority while this k-step's MFMAs issue: the SIMD's other wavefront (at a
    // barrier, its loads or its epilogue) yields the issue slots (+1-4% on dW, +0-2% on
    // dhidden; the hand-over block and a higher level measured no better)
    __builtin_amdgcn_s_setprio(1);
    frags(stage, kk_next, na, nb);
    mma(fa, fb);
    if constexpr (BKM) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 12; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
  };
  // Long-K GEMMs (dhidden, dW) hand a stage over with a split barrier on an LDS counter: a
  // wavefront arrives (adds 1) once its own loads of tile kt+1 have landed and its own reads of
  // tile kt are done, issues 16 more MFMAs, and only then waits for the count of all
  // wavefronts.  With s_barrier a wavefront can only arrive after issuing those MFMAs, and the
  // MFMA pipes drain while the last ones come in (a copy without the barrier, wrong results,
  // ran 4-13% faster); the split form measured +2-4% on these GEMMs and -3% on the short-K
  // logits GEMM, which keeps s_barrier.  The wait is bounded: running out of spins sets
  // FASTRL_SB_SYNC_TIMEOUT in the status word (the results are then not to be trusted).
  constexpr bool SPLIT = MODE != MODE_FWD;
  typedef __attribute__((address_space(3))) uint32_t lds_u32_t;
  lds_u32_t* sync = (lds_u32_t*)(smem + 2 * 2 * TILE);
  if (SPLIT && tid == 0) *sync = 0u;
  issue(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if (nk == 1 && ktail) zero_tail(0, 0);
  __syncthreads();
  frags(0, 0, fa0, fb0);
  if (nk > 1) issue(1, 1);
  // one 64-wide tile with its hand-over; LOAD: tile kt+2 exists and is loaded into the stage
  // tile kt frees (false only for the last hand-over)
  auto iteration = [&](int kt, auto load) {
    constexpr bool LOAD = decltype(load)::value;
    const int cur = kt & 1;
    kstep(cur, 1, fa0, fb0, fa1, fb1);
    // last k-step: half of its MFMAs cover the barrier; the other half cover the next
    // tile's load issue and the first fragment reads of tile kt+1
    frag_wait(fb1);
    if constexpr (SPLIT) {
      if (kt + 2 == nk && ktail) zero_tail(kt + 1, cur ^ 1);
      // own part of tile kt+1 is in LDS and own reads of tile kt are done
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      // (the add follows the first MFMA row, after the compiler's own wait for the fragments,
      // so that no wait lands between the add and the MFMAs)
      mma_rows(fa1, fb1, 0, 1);
      __builtin_amdgcn_sched_barrier(0);
      if (lane == 0) __hip_atomic_fetch_add(sync, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      __builtin_amdgcn_sched_barrier(0);
      mma_rows(fa1, fb1, 1, 2);
      __builtin_amdgcn_sched_barrier(0);
      uint32_t seen = __hip_atomic_load(sync, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      __builtin_amdgcn_sched_barrier(0);
      mma_rows(fa1, fb1, 2, 4);
      __builtin_amdgcn_sched_barrier(0);
      const uint32_t target = uint32_t(kt + 1) * (Geo<uint16_t, MODE>::THREADS / 64);
      for (int spin = 0; spin < kSyncSpins && seen < target; ++spin) {
        __builtin_amdgcn_s_sleep(0);
        seen = __hip_atomic_load(sync, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
      if (seen < target && lane == 0) set_status(p.status, FASTRL_SB_SYNC_TIMEOUT);
      asm volatile("" ::: "memory");  // LDS reads and loads of the next tile stay below
    } else {
      mma_half(fa1, fb1, 0);
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // tile kt+1 is in LDS
      if (kt + 2 == nk && ktail) zero_tail(kt + 1, cur ^ 1);
      __syncthreads();                                   // and nobody reads tile kt any more
    }
    if constexpr (LOAD) issue(kt + 2, cur);
    frags(cur ^ 1, 0, fa0, fb0);
    mma_half(fa1, fb1, 1);
    if constexpr (LOAD) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, NRD / 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, NRD / 2, 0);
    __builtin_amdgcn_sched_barrier(0);
  };
  int kt = 0;
  for (; kt + 2 < nk; ++kt) iteration(kt, std::true_type{});
  if (kt + 1 < nk) iteration(kt++, std::false_type{});
  {  // last tile
    const int cur = kt & 1;
    kstep(cur, 1, fa0, fb0, fa1, fb1);
    frag_wait(fb1);
    mma(fa1, fb1);
  }
}

// float32 main loop (small problems): register-staged loads into padded LDS rows.  With
// A_KMAJOR the A operand is stored k-major (A[m][k] at k * lda + m): a thread loads 4
// consecutive m of one k and scatters them into the tile's rows.
template <int MODE, bool A_KMAJOR>
__device__ __forceinline__ void mainloop_f32(const GemmParams& p, int m0, int n0,
                                             f32x16_t (&acc)[4][4], float* smem) {
  using E = Eng<float>;
  constexpr int BK = E::BK, LD = E::LD, VEC = E::VEC;
  constexpr int VPR = BK / VEC;
  constexpr int LOADS = kBM * VPR / Geo<float, MODE>::THREADS;
  float* As = smem;
  float* Bs = smem + 2 * kBM * LD;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const float* Ag = static_cast<const float*>(p.A);
  const float* Bg = static_cast<const float*>(p.B);
  const float* arow[LOADS];
  const float* brow[LOADS];
  bool aok[LOADS], bok[LOADS];
  int kofs[LOADS], srow[LOADS], akk[LOADS], am4[LOADS];
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int v = tid + j * Geo<float, MODE>::THREADS;
    const int row = v / VPR;
    kofs[j] = (v % VPR) * VEC;
    srow[j] = row;
    const int am = m0 + row;
    aok[j] = am < p.M;
    arow[j] = Ag + int64_t(aok[j] ? am : 0) * p.lda;
    akk[j] = v / (kBM / VEC);         // k-major: k row of the tile
    am4[j] = (v % (kBM / VEC)) * VEC;  // and 4 consecutive m
    const int bn = n0 + row;
    bok[j] = bn < p.N;
    int64_t br = bok[j] ? bn : 0;
    if (MODE == MODE_FWD) {
      br += p.b_row_base;
      if (p.b_rows) br = bok[j] ? p.b_rows[br] : 0;
    }
    brow[j] = Bg + br * p.ldb;
  }
  u32x4_t ra[LOADS], rb[LOADS];
  const int nk = (p.K + BK - 1) / BK;
  auto gload = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      const int k = k0 + kofs[j];
      if (A_KMAJOR) {
        const int ka = k0 + akk[j];
        const int mm = m0 + am4[j];
        load_vec<float>(Ag + int64_t(ka) * p.lda + mm, ka < p.K && mm + VEC <= p.lda, ra[j]);
      } else {
        load_vec<float>(arow[j] + k, aok[j] && k < p.K, ra[j]);
      }
      load_vec<float>(brow[j] + k, bok[j] && k < p.K, rb[j]);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      if (A_KMAJOR) {
#pragma unroll
        for (int q = 0; q < VEC; ++q)
          As[(buf * kBM + am4[j] + q) * LD + akk[j]] = __uint_as_float(ra[j][q]);
      } else {
        *reinterpret_cast<u32x4_t*>(As + (buf * kBM + srow[j]) * LD + kofs[j]) = ra[j];
      }
      *reinterpret_cast<u32x4_t*>(Bs + (buf * kBM + srow[j]) * LD + kofs[j]) = rb[j];
    }
  };
  gload(0);
  sstore(0);
  for (int kt = 0; kt < nk; ++kt) {
    __syncthreads();
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const float* as = As + buf * kBM * LD;
    const float* bs = Bs + buf * kBM * LD;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
      float af[4], bf[4];
      const int kq = kk + (lane >> 5);
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = as[(wm * 128 + i * 32 + (lane & 31)) * LD + kq];
#pragma unroll
      for (int j = 0; j < 4; ++j) bf[j] = bs[(wn * 128 + j * 32 + (lane & 31)) * LD + kq];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
  }
}


// Reductions over the four 16-lane groups of a wavefront (lanes c, c + 16, c + 32, c + 48) with
// row swaps instead of LDS-routed shuffles: a 16-lane-row swap of x with itself leaves rows
// (r0, r0, r2, r2) and (r1, r1, r3, r3), whose sum is the xor-16 partner sum; a half swap then
// does the same for xor 32.  Each step adds the same two operands as the xor shuffle would.
__device__ __forceinline__ float group_sum4(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ float group_max4(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Epilogue of the bf16 logits GEMM (16 x 16 accumulator tiles: acc[i][j] covers vocab rows
// wm*128 + 16 i .. +15 and tokens wn*64 + 16 j .. +15; lane l holds rows 4 (l / 16) + q of
// token column l % 16).  Per token column: the block's max over its vocab rows, the sampled
// token's logit, and with a stored exp (store_e != 0) E[t][v] = exp(z - s_t) with the sums
// sum exp(z - s_t) and sum exp(z - s_t) z; without one (old / ref log-probs), the sums relative
// to the block max.  A column's 256 rows are spread over the 4 lane groups of two wavefronts:
// lane-row swaps, then one LDS exchange between the wavefronts.
__device__ __forceinline__ void fwd_epilogue_bf16(const GemmParams& p, int m0, int n0, int mb,
                                                  f32x4_t (&acc)[8][4], uint16_t* smem) {
  __syncthreads();  // LDS operand buffers are reused for the cross-wave exchange
  float* xmax = reinterpret_cast<float*>(smem);  // [2 wm][256 cols]
  float* xsum = xmax + 2 * kBN;
  float* xsz = xsum + 2 * kBN;
  constexpr int NT = Geo<uint16_t, MODE_FWD>::THREADS;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int g = lane >> 4, c = lane & 15;
  const int Vr = p.Vreal;
  const bool rel = p.store_e != 0;
  const bool rows_full = m0 + kBM <= Vr;  // every vocab row of this block exists
  const int rbase = m0 + wm * 128 + 4 * g;  // vocab row of acc[i][j][q]: rbase + 16 i + q
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int cl = wn * 64 + j * 16 + c;
    const int t = n0 + cl;  // slab token
    const bool tok_ok = t < p.N;
    const int y = tok_ok ? p.yslab[t] : -1;
    // columns past the slab store exp(z - inf) = 0
    const float s_t = tok_ok ? (p.shift ? p.shift[t] : 0.0f) : INFINITY;
    // max over the lane's 32 rows in four independent chains; a full vocab block (all but the
    // last) takes a branch without the row test, so the chains become three-input maxima
    float mxp[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    if (rows_full) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) mxp[i & 3] = fmaxf(mxp[i & 3], acc[i][j][q]);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          mxp[i & 3] = fmaxf(mxp[i & 3], rbase + 16 * i + q < Vr ? acc[i][j][q] : -INFINITY);
    }
    float mx = fmaxf(fmaxf(mxp[0], mxp[1]), fmaxf(mxp[2], mxp[3]));
    // the sampled token's logit: held by one lane group of one wavefront (rare per column)
    const int dy = y - m0 - wm * 128;
    if (dy >= 0 && dy < 128 && ((dy >> 2) & 3) == g) {
      float zl = 0.0f;
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) zl = (16 * i + q == (dy & ~12)) ? acc[i][j][q] : zl;
      p.zlab[t] = zl;
    }
    mx = group_max4(mx);
    if (g == 0) xmax[wm * kBN + cl] = mx;
    if (rel) {
      uint16_t* e1 = static_cast<uint16_t*>(p.E1) + int64_t(t) * p.ldE1;
      // exp(z - s_t) = exp2(z log2e - s_t log2e): one FMA and v_exp_f32 per logit (s_t = +inf
      // past the slab gives 0).  Two uniform choices get code of their own, since this pass is
      // most of the epilogue (a per-block timing probe: 8.5% of the kernel): the row check only
      // in the last vocab block, the z-weighted sum only when the entropy is asked for.
      const float sl = s_t * 1.4426950408889634f;
      auto pass = [&](auto full_c, auto z_c) {
        constexpr bool FULL = decltype(full_c)::value, WZ = decltype(z_c)::value;
        float ssp[4] = {0.0f, 0.0f, 0.0f, 0.0f}, zsp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ip = 0; ip < 4; ++ip) {  // tile pair 2 ip, 2 ip + 1
          uint32_t pk[2][2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int i = 2 * ip + h;
            float e[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              e[q] = __builtin_amdgcn_exp2f(fmaf(acc[i][j][q], 1.4426950408889634f, -sl));
              if (!FULL && rbase + 16 * i + q >= Vr) e[q] = 0.0f;
              ssp[ip] += e[q];
              if (WZ) zsp[ip] = fmaf(e[q], acc[i][j][q], zsp[ip]);
            }
            typedef float f32x2_t __attribute__((ext_vector_type(2)));
            typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
            pk[h][0] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{e[0], e[1]}, bf16x2_t));
            pk[h][1] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{e[2], e[3]}, bf16x2_t));
          }
          // lane group g holds rows 4 g .. 4 g + 3 of both tiles; one swap between the groups
          // of each 32-lane half (odd group's tile-2ip rows <-> even group's tile-2ip+1 rows)
          // leaves group g with 8 consecutive rows: tile 2 ip + (g & 1), rows 8 (g >> 1) .. + 7
#pragma unroll
          for (int w = 0; w < 2; ++w) {
            const auto sw = __builtin_amdgcn_permlane16_swap(pk[0][w], pk[1][w], false, false);
            pk[0][w] = sw[0];
            pk[1][w] = sw[1];
          }
          const int v0 = m0 + wm * 128 + (2 * ip + (g & 1)) * 16 + (g >> 1) * 8;
          *reinterpret_cast<uint4*>(e1 + v0) = make_uint4(pk[0][0], pk[0][1], pk[1][0], pk[1][1]);
        }
        float ssum = (ssp[0] + ssp[1]) + (ssp[2] + ssp[3]);
        ssum = group_sum4(ssum);
        if (g == 0) xsum[wm * kBN + cl] = ssum;
        if constexpr (WZ) {
          float zsum = (zsp[0] + zsp[1]) + (zsp[2] + zsp[3]);
          zsum = group_sum4(zsum);
          if (g == 0) xsz[wm * kBN + cl] = zsum;
        }
      };
      if (rows_full) {
        if (p.psz) pass(std::true_type{}, std::true_type{});
        else pass(std::true_type{}, std::false_type{});
      } else {
        if (p.psz) pass(std::false_type{}, std::true_type{});
        else pass(std::false_type{}, std::false_type{});
      }
    }
  }
  __syncthreads();
  if (!rel) {
    // sums relative to the block's column max M: exp(z - M) = exp2(z log2e - M log2e), one FMA
    // and one v_exp_f32 per logit; as in the stored-exp pass, full vocab blocks skip the row
    // test and the z-weighted sum is only formed when the entropy is asked for
    auto pass = [&](auto full_c, auto z_c) {
      constexpr bool FULL = decltype(full_c)::value, WZ = decltype(z_c)::value;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int cl = wn * 64 + j * 16 + c;
        const float ml = fmaxf(xmax[cl], xmax[kBN + cl]) * 1.4426950408889634f;
        float ssp[4] = {0.0f, 0.0f, 0.0f, 0.0f}, zsp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float ex = __builtin_amdgcn_exp2f(fmaf(acc[i][j][q], 1.4426950408889634f, -ml));
            if (!FULL && rbase + 16 * i + q >= Vr) ex = 0.0f;
            ssp[i & 3] += ex;
            if (WZ) zsp[i & 3] = fmaf(ex, acc[i][j][q], zsp[i & 3]);
          }
        float ssum = (ssp[0] + ssp[1]) + (ssp[2] + ssp[3]);
        ssum = group_sum4(ssum);
        if (g == 0) xsum[wm * kBN + cl] = ssum;
        if constexpr (WZ) {
          float zsum = (zsp[0] + zsp[1]) + (zsp[2] + zsp[3]);
          zsum = group_sum4(zsum);
          if (g == 0) xsz[wm * kBN + cl] = zsum;
        }
      }
    };
    if (rows_full) {
      if (p.psz) pass(std::true_type{}, std::true_type{});
      else pass(std::true_type{}, std::false_type{});
    } else {
      if (p.psz) pass(std::false_type{}, std::true_type{});
      else pass(std::false_type{}, std::false_type{});
    }
    __syncthreads();
  }
  for (int cl = tid; cl < kBN; cl += NT) {
    const int t = n0 + cl;
    if (t < p.N) {
      p.pmax[int64_t(mb) * p.ldp + t] = fmaxf(xmax[cl], xmax[kBN + cl]);
      p.psum[int64_t(mb) * p.ldp + t] = xsum[cl] + xsum[kBN + cl];
      if (p.psz) p.psz[int64_t(mb) * p.ldp + t] = xsz[cl] + xsz[kBN + cl];
    }
  }
}


// Epilogue of the bf16 dhidden GEMM on the 16 x 16 layout (acc[i][j]: token rows wm*128 + 16 i
// + 4 (l / 16) + q, hidden columns wn*64 + 16 j + l % 16): dH[t] = -c_t C[t] (the one-hot term
// is already in E1).
__device__ __forceinline__ void dh_epilogue_bf16(const GemmParams& p, int m0, int n0,
                                                 f32x4_t (&acc)[8][4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int g = lane >> 4, c = lane & 15;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int t = m0 + wm * 128 + 16 * i + 4 * g + q;
      if (t < p.M) {
        const float ct = p.cslab[t];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = n0 + wn * 64 + 16 * j + c;
          if (n < p.N) {
            const float val = -ct * acc[i][j][q];
            const int64_t o = int64_t(t) * p.d + n;
            if (p.dH_bf16) static_cast<uint16_t*>(p.dH)[o] = f32_to_bf16(val);
            else static_cast<float*>(p.dH)[o] = val;
          }
        }
      }
    }
}

// Epilogue of the bf16 dW GEMM computed transposed (C' = Bd E on the 16 x 16 layout: acc[i][j]
// holds hidden columns n = wm*128 + 16 i + 4 (l / 16) + q of vocab row v = wn*64 + 16 j + l % 16):
// each lane owns 4 consecutive n of one dW row and moves them as one 16-byte access.
// dW[v][n] (+)= -C'[n][v] (the one-hot term is already in E1).  Needs d % 4 == 0 and a 16-byte
// aligned dW (checked on the host).
__device__ __forceinline__ void dwt_epilogue_bf16(const GemmParams& p, int m0, int n0,
                                                  f32x4_t (&acc)[8][4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int nq = m0 + wm * 128 + 4 * (lane >> 4);  // first hidden column of acc[0][j]
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = n0 + wn * 64 + 16 * j + (lane & 15);
    if (v < p.N) {
      f32x4_t* row = reinterpret_cast<f32x4_t*>(p.dW + int64_t(v) * p.d);
      // every load of the row first, so that their latencies overlap
      f32x4_t prev[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int n = nq + 16 * i;
        prev[i] = (p.dW_acc && n < p.M) ? row[n >> 2] : f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int n = nq + 16 * i;
        if (n < p.M) row[n >> 2] = prev[i] - acc[i][j];
      }
    }
  }
}

template <typename T>
struct SmemBytes;
template <>
struct SmemBytes<uint16_t> { static constexpr int value = 2 * 2 * kBM * 64 * 2 + 16; };  // + sync word
template <>
struct SmemBytes<float> { static constexpr int value = 2 * 2 * kBM * Eng<float>::LD * 4; };

template <typename T, int MODE>
__global__ __launch_bounds__((Geo<T, MODE>::THREADS))
__attribute__((amdgpu_waves_per_eu(Geo<T, MODE>::WPE, Geo<T, MODE>::WPE)))
void lm_gemm_kernel(const GemmParams p) {
  __shared__ __attribute__((aligned(16))) char smem_raw[SmemBytes<T>::value];
  T* smem = reinterpret_cast<T*>(smem_raw);
  int mb, nb;
  tile_coords<MODE>(mb, nb, p.nmb, p.nnb, blockIdx.x, p.group);
  if (MODE == MODE_FWD && p.store_e == 2 && p.redo_blk[nb] == 0) return;
  const int m0 = mb * kBM, n0 = nb * kBN;
  constexpr int NI = Geo<T, MODE>::NI, NT = Geo<T, MODE>::THREADS;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / Geo<T, MODE>::WAVES_N, wn = wave % Geo<T, MODE>::WAVES_N;

  if constexpr (Geo<T, MODE>::W8) {
    f32x4_t acc16[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc16[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    mainloop_bf16_dma<MODE>(p, m0, n0, acc16, smem);
    if constexpr (MODE == MODE_FWD) fwd_epilogue_bf16(p, m0, n0, mb, acc16, smem);
    else if constexpr (MODE == MODE_DH) dh_epilogue_bf16(p, m0, n0, acc16);
    else dwt_epilogue_bf16(p, m0, n0, acc16);
    return;
  }
  f32x16_t acc[4][NI];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = f32x16_t{};
  if constexpr (sizeof(T) == 4) mainloop_f32<MODE, MODE == MODE_DW>(p, m0, n0, acc, smem);

  // ------------------------------------------------------------------ epilogues
  if constexpr (MODE == MODE_FWD && sizeof(T) == 4) {  // float32 logits (bf16: fwd_epilogue_bf16)
    __syncthreads();  // LDS operand buffers are reused for the cross-wave exchange
    float* xmax = reinterpret_cast<float*>(smem);      // [2 wm][256 cols]
    float* xsum = xmax + 2 * kBN;
    float* xsz = xsum + 2 * kBN;
    const int Vr = p.Vreal;
    // with a stored exp (store_e != 0) the block's sum is taken relative to the row's shift
    // s_t, sum_v exp(z - s_t): one exp per logit serves both the sum and the stored E.  The
    // merge checks that max_t - s_t stays inside (-60, 60) and re-runs rows that do not.
    const bool rel = p.store_e != 0;
    const bool rows_full = m0 + kBM <= Vr;  // every vocab row of this block exists
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
      const int cl = acc_col<T, MODE>(wn, ni, lane);
      const int t = n0 + cl;                 // slab token
      const bool tok_ok = t < p.N;
      const int y = tok_ok ? p.yslab[t] : -1;
      // columns past the slab store exp(z - inf) = 0
      const float s_t = tok_ok ? (p.shift ? p.shift[t] : 0.0f) : INFINITY;
      // four independent chains (one per 32-row group), combined at the end
      float mxp[4];
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        mxp[mi] = -INFINITY;
        if (rows_full) {
#pragma unroll
          for (int r = 0; r < 16; ++r) mxp[mi] = fmaxf(mxp[mi], acc[mi][ni][r]);
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r)
            mxp[mi] = (m0 + acc_row(wm, mi, r, lane) < Vr) ? fmaxf(mxp[mi], acc[mi][ni][r]) : mxp[mi];
        }
      }
      float mx = fmaxf(fmaxf(mxp[0], mxp[1]), fmaxf(mxp[2], mxp[3]));
      // the sampled token's logit: held by one lane half of one wavefront (rare per column)
      const int dy = y - m0 - wm * 128;
      if (dy >= 0 && dy < 128 && ((dy >> 2) & 1) == (lane >> 5)) {
        float zl = 0.0f;
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            zl = (mi * 32 + (r >> 2) * 8 + (r & 3) == (dy & ~4)) ? acc[mi][ni][r] : zl;
        p.zlab[t] = zl;
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (lane < 32) xmax[wm * kBN + cl] = mx;
      if (rel) {
        // sum exp(z - s_t) and sum exp(z - s_t) z, one chain per 32-row group
        float ssp[4] = {0.0f, 0.0f, 0.0f, 0.0f}, zsp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        T* e1 = static_cast<T*>(p.E1) + int64_t(t) * p.ldE1;
#pragma unroll
        for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
          for (int rg = 0; rg < 4; ++rg) {
            float e[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              e[q] = __expf(acc[mi][ni][rg * 4 + q] - s_t);
              if (!rows_full && m0 + acc_row(wm, mi, rg * 4 + q, lane) >= Vr) e[q] = 0.0f;
              ssp[mi] += e[q];
              zsp[mi] = fmaf(e[q], acc[mi][ni][rg * 4 + q], zsp[mi]);
            }
            const int v0 = m0 + acc_row(wm, mi, rg * 4, lane);
            *reinterpret_cast<float4*>(e1 + v0) = make_float4(e[0], e[1], e[2], e[3]);
          }
        }
        float ssum = (ssp[0] + ssp[1]) + (ssp[2] + ssp[3]);
        float zsum = (zsp[0] + zsp[1]) + (zsp[2] + zsp[3]);
        ssum += __shfl_xor(ssum, 32, 64);
        zsum += __shfl_xor(zsum, 32, 64);
        if (lane < 32) {
          xsum[wm * kBN + cl] = ssum;
          xsz[wm * kBN + cl] = zsum;
        }
      }
    }
    __syncthreads();
    if (!rel) {
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) {
        const int cl = acc_col<T, MODE>(wn, ni, lane);
        const float M = fmaxf(xmax[cl], xmax[kBN + cl]);
        float ssp[4] = {0.0f, 0.0f, 0.0f, 0.0f}, zsp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int v = m0 + acc_row(wm, mi, r, lane);
            if (v < Vr) {
              const float ex = __expf(acc[mi][ni][r] - M);
              ssp[mi] += ex;
              zsp[mi] = fmaf(ex, acc[mi][ni][r], zsp[mi]);
            }
          }
        float ssum = (ssp[0] + ssp[1]) + (ssp[2] + ssp[3]);
        float zsum = (zsp[0] + zsp[1]) + (zsp[2] + zsp[3]);
        ssum += __shfl_xor(ssum, 32, 64);
        zsum += __shfl_xor(zsum, 32, 64);
        if (lane < 32) {
          xsum[wm * kBN + cl] = ssum;
          xsz[wm * kBN + cl] = zsum;
        }
      }
      __syncthreads();
    }
    for (int cl = tid; cl < kBN; cl += NT) {
      const int t = n0 + cl;
      if (t < p.N) {
        p.pmax[int64_t(mb) * p.ldp + t] = fmaxf(xmax[cl], xmax[kBN + cl]);
        p.psum[int64_t(mb) * p.ldp + t] = xsum[cl] + xsum[kBN + cl];
        if (p.psz) p.psz[int64_t(mb) * p.ldp + t] = xsz[cl] + xsz[kBN + cl];
      }
    }
  } else if constexpr (MODE == MODE_DH && !Geo<T, MODE>::W8) {  // dH[t] = -c_t C[t]
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int t = m0 + acc_row(wm, mi, r, lane);
        if (t < p.M) {
          const float c = p.cslab[t];
#pragma unroll
          for (int ni = 0; ni < NI; ++ni) {
            const int n = n0 + acc_col<T, MODE>(wn, ni, lane);
            if (n < p.N) {
              const float val = -c * acc[mi][ni][r];
              const int64_t o = int64_t(t) * p.d + n;
              if (p.dH_bf16) static_cast<uint16_t*>(p.dH)[o] = f32_to_bf16(val);
              else static_cast<float*>(p.dH)[o] = val;
            }
          }
        }
      }
  } else {  // MODE_DW: dW[v] (+)= -C[v] (the one-hot term is already in E1)
    // RB rows at a time
    constexpr int RB = 4;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int rh = 0; rh < 16; rh += RB) {
        // every load of these rows first, so that their latencies overlap
        float prev[RB][NI];
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          const int v = m0 + acc_row(wm, mi, rh + r, lane);
#pragma unroll
          for (int ni = 0; ni < NI; ++ni) {
            const int n = n0 + acc_col<T, MODE>(wn, ni, lane);
            prev[r][ni] = (p.dW_acc && v < p.M && n < p.N) ? p.dW[int64_t(v) * p.d + n] : 0.0f;
          }
        }
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          const int v = m0 + acc_row(wm, mi, rh + r, lane);
#pragma unroll
          for (int ni = 0; ni < NI; ++ni) {
            const int n = n0 + acc_col<T, MODE>(wn, ni, lane);
            if (v < p.M && n < p.N) p.dW[int64_t(v) * p.d + n] = prev[r][ni] - acc[mi][ni][rh + r];
          }
        }
      }
  }
}

// The two bf16 backward GEMMs of one slab in one launch: blocks [0, q.nmb q.nnb) are dhidden
// tiles (K = padded vocabulary), the rest transposed-dW tiles (K = padded slab, about five times
// shorter at the 7B shape).  Dispatched in block order, the dW tiles take the compute units that
// the last partial wave of dhidden tiles leaves idle (a 27K-token slab has 5.8 waves of
// dhidden tiles, a 19K-token slab at d = 1536 only 1.7).
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void lm_bwd_kernel(const GemmParams q, const GemmParams r) {
  __shared__ __attribute__((aligned(16))) char smem_raw[SmemBytes<uint16_t>::value];
  uint16_t* smem = reinterpret_cast<uint16_t*>(smem_raw);
  const int nh = q.nmb * q.nnb;
  const int b = blockIdx.x;
  int mb, nb;
  f32x4_t acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  if (b < nh) {
    tile_coords<MODE_DH>(mb, nb, q.nmb, q.nnb, b, q.group);
    mainloop_bf16_dma<MODE_DH>(q, mb * kBM, nb * kBN, acc, smem);
    dh_epilogue_bf16(q, mb * kBM, nb * kBN, acc);
  } else {
    tile_coords<MODE_DWT>(mb, nb, r.nmb, r.nnb, b - nh, r.group);
    mainloop_bf16_dma<MODE_DWT>(r, mb * kBM, nb * kBN, acc, smem);
    dwt_epilogue_bf16(r, mb * kBM, nb * kBN, acc);
  }
}

// Second evaluation of the bf16 logits tiles whose token block holds a row that needs a shift:
// at most one block per compute unit walks the tiles in grid order and evaluates those of marked
// token blocks (store_e == 2); with no row marked, the usual case, every block returns at once.
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void lm_redo_kernel(const GemmParams p) {
  if (p.redo_any[0] == 0) return;
  __shared__ __attribute__((aligned(16))) char smem_raw[SmemBytes<uint16_t>::value];
  uint16_t* smem = reinterpret_cast<uint16_t*>(smem_raw);
  const int nt = p.nmb * p.nnb;
  for (int b = blockIdx.x; b < nt; b += gridDim.x) {
    int mb, nb;
    tile_coords<MODE_FWD>(mb, nb, p.nmb, p.nnb, b, p.group);
    if (p.redo_blk[nb] == 0) continue;  // the same for the whole block
    f32x4_t acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    mainloop_bf16_dma<MODE_FWD>(p, mb * kBM, nb * kBN, acc, smem);
    fwd_epilogue_bf16(p, mb * kBM, nb * kBN, mb, acc, smem);
    __syncthreads();  // the epilogue's LDS exchange is read before the next tile's loads land
  }
}

// ------------------------------------------------------------------ small kernels

// s_t = 0, labels of the slab, validity
__global__ void slab_prep_kernel(const int32_t* __restrict__ token_ids,
                                 const int32_t* __restrict__ row_index, int64_t row_base,
                                 int32_t Tc, int32_t V, int32_t* __restrict__ yslab,
                                 float* __restrict__ shift, int32_t* __restrict__ status) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Tc) return;
  int64_t row = row_base + t;
  if (row_index) row = row_index[row];
  int y = token_ids[row];
  if (y < 0 || y >= V) {
    set_status(status, FASTRL_SB_BAD_TOKEN);
    y = -1;
  }
  yslab[t] = y;
  if (shift) shift[t] = 0.0f;
}

// partials -> lse, logp.  One block of 256 threads handles 64 tokens; its 4 wavefronts
// each combine a quarter of the vocabulary blocks, then combine through LDS.
//   rel == 0: psum = sum exp(z - pmax) per vocab block (log-prob only path)
//   rel == 1: psum = sum exp(z - s_t); with check != 0 a row whose max is too far from s_t
//             (exp(z - s_t) could leave float range) gets s_t = max and its token block is
//             marked for a second evaluation.
__global__ __launch_bounds__(256) void merge_kernel(
    const float* __restrict__ pmax, const float* __restrict__ psum,
    const float* __restrict__ psz, int64_t ldp, int32_t nmb, const float* __restrict__ zlab,
    const int32_t* __restrict__ yslab, int32_t Tc, int32_t rel, int32_t check,
    float* __restrict__ lse_out, float* __restrict__ logp_out, float* __restrict__ ent_out,
    float* __restrict__ shift, int32_t* __restrict__ redo_blk, int32_t* __restrict__ redo_count,
    int32_t* __restrict__ redo_any, int32_t only_after_redo) {
  // the second merge only matters when the first marked a row (every block reads the same flag)
  if (only_after_redo && redo_any[0] == 0) return;
  __shared__ float sm[4][64], ss[4][64], sz[4][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int t = blockIdx.x * 64 + lane;
  const bool ok = t < Tc;
  const bool ent = psz != nullptr;
  // S = sum exp(z - ref), Z = sum exp(z - ref) z, both relative to the same reference
  float M = -INFINITY, S = 0.0f, Z = 0.0f;
  if (ok) {
    for (int b = wv; b < nmb; b += 4) {
      const float m = pmax[int64_t(b) * ldp + t];
      const float x = psum[int64_t(b) * ldp + t];
      const float y = ent ? psz[int64_t(b) * ldp + t] : 0.0f;
      if (rel) {
        M = fmaxf(M, m);
        S += x;
        Z += y;
      } else if (m > M) {
        const float f = __expf(M - m);
        S = S * f + x;
        Z = Z * f + y;
        M = m;
      } else {
        const float f = __expf(m - M);
        S += x * f;
        Z += y * f;
      }
    }
  }
  sm[wv][lane] = M;
  ss[wv][lane] = S;
  sz[wv][lane] = Z;
  __syncthreads();
  if (wv != 0 || !ok) return;
  float Mt = sm[0][lane], St = ss[0][lane], Zt = sz[0][lane];
  for (int w = 1; w < 4; ++w) {
    const float m = sm[w][lane], x = ss[w][lane], y = sz[w][lane];
    if (rel) {
      Mt = fmaxf(Mt, m);
      St += x;
      Zt += y;
    } else if (m > Mt) {
      const float f = __expf(Mt - m);
      St = St * f + x;
      Zt = Zt * f + y;
      Mt = m;
    } else if (m > -INFINITY) {
      const float f = __expf(m - Mt);
      St += x * f;
      Zt += y * f;
    }
  }
  const float s_t = (rel && shift) ? shift[t] : 0.0f;
  const float l = rel ? s_t + __logf(St) : Mt + __logf(St);
  const int y = yslab[t];
  if (lse_out) lse_out[t] = l;
  if (logp_out) logp_out[t] = y >= 0 ? zlab[t] - l : __int_as_float(0x7fc00000);
  // entropy -sum_v p_v log p_v = lse - sum_v p_v z_v, sum_v p_v z_v = Z / S
  if (ent_out) ent_out[t] = l - Zt / St;
  if (rel && check && !(Mt - s_t < 60.0f && Mt - s_t > -60.0f)) {
    shift[t] = Mt;
    redo_blk[t / kBN] = 1;
    redo_any[0] = 1;
    atomicAdd(redo_count, 1);
  }
}

// sum of x[0..n) in float64, fixed order (one block): the mean entropy of the kept tokens
__global__ __launch_bounds__(256) void sum_f32_kernel(const float* __restrict__ x, int64_t n,
                                                      float* __restrict__ out) {
  __shared__ double red[4];
  double s = 0.0;
  const int64_t per = (n + blockDim.x - 1) / blockDim.x;
  const int64_t b = threadIdx.x * per, e = min(n, b + per);
  for (int64_t i = b; i < e; ++i) s += double(x[i]);
  // fixed-shape tree: wave butterfly, then the 4 wave sums in order
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) red[wv] = s;
  __syncthreads();
  if (threadIdx.x == 0) out[0] = float(((red[0] + red[1]) + red[2]) + red[3]);
}

__device__ __forceinline__ double block_sum_d(double v, double* red) {
  // fixed-shape tree: wave butterfly, then the 4 wave sums in order
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  double s = 0.0;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) s += red[w];
  return s;
}

// one block per sequence of the slab: g_t, c_t, the sequence's loss term and, with a backward,
// the one-hot term of each token folded into its exp-logit row
__global__ __launch_bounds__(256) void loss_kernel(
    const float* __restrict__ logp, const float* __restrict__ lse,
    const float* __restrict__ old_logp, const float* __restrict__ ref_logp,
    const int32_t* __restrict__ row_index, const int64_t* __restrict__ seq_off,
    const float* __restrict__ adv, const int32_t* __restrict__ seq_index, int32_t S,
    int64_t T, int32_t seq_begin, int64_t row_base, int32_t algo, int32_t norm,
    float eps_low, float eps_high, float beta, const float* __restrict__ shift,
    float* __restrict__ cslab, double* __restrict__ seq_loss,
    int32_t* __restrict__ seq_clip, int32_t* __restrict__ status, int32_t nadv,
    void* __restrict__ E1, int64_t ldE1, int32_t e_bf16, const int32_t* __restrict__ yslab) {
  __shared__ double red[4];
  __shared__ double redc[4];
  const int i = seq_begin + blockIdx.x;
  const int64_t a = seq_off[i], b = seq_off[i + 1];
  const int64_t L = b - a;
  int ai = seq_index ? seq_index[i] : i;
  if (ai < 0 || ai >= nadv) {
    if (threadIdx.x == 0) set_status(status, FASTRL_SB_BAD_INDEX);
    ai = -1;
  }
  const double A = ai >= 0 ? double(adv[ai]) : 0.0;
  const double w = (norm == FASTRL_NORM_TOKEN_MEAN) ? 1.0 / double(T)
                                                    : (L > 0 ? 1.0 / (double(S) * double(L)) : 0.0);
  const double lo = 1.0 - double(eps_low), hi = 1.0 + double(eps_high);
  const bool kl = beta != 0.0f;
  double part = 0.0;  // this sequence's contribution to the loss
  int clip = 0;
  double sratio = 0.0, cseq = 0.0;
  if (algo == FASTRL_GSPO && L > 0) {
    double sl = 0.0;
    for (int64_t t = a + threadIdx.x; t < b; t += blockDim.x) {
      int64_t row = t;
      if (row_index) row = row_index[t];
      sl += double(logp[t]) - double(old_logp[row]);
    }
    sl = block_sum_d(sl, red);
    sratio = exp(sl / double(L));
    const double sur = fmin(sratio * A, fmin(fmax(sratio, lo), hi) * A);
    cseq = ((A >= 0.0 && sratio <= hi) || (A < 0.0 && sratio >= lo)) ? 1.0 : 0.0;
    if (threadIdx.x == 0) part = -(w * double(L)) * sur;
    clip = (cseq == 0.0) ? int(L) : 0;
  }
  double kpart = 0.0;
  for (int64_t t = a + threadIdx.x; t < b; t += blockDim.x) {
    int64_t row = t;
    if (row_index) row = row_index[t];
    const double x = logp[t];
    double g;
    if (algo == FASTRL_GSPO) {
      g = (w * double(L)) * (-cseq * sratio * A / double(L));
    } else {
      const double rho = exp(x - double(old_logp[row]));
      const double sur = fmin(rho * A, fmin(fmax(rho, lo), hi) * A);
      const double c = ((A >= 0.0 && rho <= hi) || (A < 0.0 && rho >= lo)) ? 1.0 : 0.0;
      kpart += -w * sur;
      g = w * (-c * rho * A);
      clip += (c == 0.0);
    }
    if (kl) {
      const double f = ref_logp[row];
      const double e = exp(f - x);
      kpart += double(beta) * w * (e - (f - x) - 1.0);
      g += double(beta) * w * (1.0 - e);
    }
    const int64_t tl = t - row_base;
    const float s_t = shift ? shift[tl] : 0.0f;
    cslab[tl] = float(g * exp(double(s_t) - double(lse[t])));
    // one-hot term of dZ folded into the exp-logits for the backward GEMMs: with
    // g_t = c_t exp(lse_t - s_t), c_t (E1[t][y_t] - exp(lse_t - s_t)) = c_t E1[t][y_t] - g_t
    const int y = E1 ? yslab[tl] : -1;
    if (y >= 0) {
      const double corr = exp(double(lse[t]) - double(s_t));
      const int64_t o = tl * ldE1 + y;
      if (e_bf16) {
        uint16_t* e = static_cast<uint16_t*>(E1) + o;
        *e = f32_to_bf16(float(double(bf16_to_f32(*e)) - corr));
      } else {
        float* e = static_cast<float*>(E1) + o;
        *e = float(double(*e) - corr);
      }
    }
  }
  kpart = block_sum_d(kpart, red);
  const double clips = block_sum_d(algo == FASTRL_GSPO ? 0.0 : double(clip), redc);
  if (threadIdx.x == 0) {
    seq_loss[i] = part + kpart;
    seq_clip[i] = algo == FASTRL_GSPO ? clip : int(clips);
  }
}

// sum of per-sequence loss terms in index order (deterministic)
__global__ void loss_final_kernel(const double* __restrict__ seq_loss,
                                  const int32_t* __restrict__ seq_clip, int32_t S,
                                  const int32_t* __restrict__ redo_count,
                                  float* __restrict__ loss, float* __restrict__ stats) {
  __shared__ double red[4];
  __shared__ double redc[4];
  double s = 0.0, c = 0.0;
  // contiguous chunk per thread keeps the order fixed for a given S
  const int per = (S + blockDim.x - 1) / blockDim.x;
  const int b = threadIdx.x * per, e = min(S, b + per);
  for (int i = b; i < e; ++i) {
    s += seq_loss[i];
    c += seq_clip[i];
  }
  s = block_sum_d(s, red);
  c = block_sum_d(c, redc);
  if (threadIdx.x == 0) {
    loss[0] = float(s);
    if (stats) {
      stats[0] = float(c);
      stats[1] = float(redo_count[0]);
    }
  }
}

// out[c][r] = scale(r) * in[row(r)][c], zero for r in [R, Rpad): 64 x 64 tiles through LDS with
// 16-byte global loads and stores (C is a multiple of 8, in 16-byte aligned, Rpad and ldo
// multiples of 64, out 256-byte aligned)
template <typename T>
__global__ __launch_bounds__(256) void transpose_scale_kernel(
    const T* __restrict__ in, const int32_t* __restrict__ row_index, int64_t row_base,
    int32_t R, int32_t Rpad, int32_t C, const float* __restrict__ scale, T* __restrict__ out,
    int64_t ldo) {
  constexpr int VEC = 16 / sizeof(T);  // elements per 16-byte piece: 8 bf16 or 4 float
  constexpr int LPR = 64 / VEC;        // threads per 64-element tile row
  constexpr int RPP = 256 / LPR;       // tile rows per pass
  __shared__ float tile[64][65];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tid = threadIdx.x;
  const int l = (tid % LPR) * VEC;
  for (int rr = tid / LPR; rr < 64; rr += RPP) {
    const int r = r0 + rr;
    float v[VEC];
    if (r < R && c0 + l < C) {
      int64_t row = row_base + r;
      if (row_index) row = row_index[row];
      const u32x4_t raw = *reinterpret_cast<const u32x4_t*>(in + row * C + c0 + l);
      const float sc = scale ? scale[r] : 1.0f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (sizeof(T) == 2) {
          v[2 * q] = bf16_to_f32(uint16_t(raw[q] & 0xffffu)) * sc;
          v[2 * q + 1] = bf16_to_f32(uint16_t(raw[q] >> 16)) * sc;
        } else {
          v[q] = __uint_as_float(raw[q]) * sc;
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < VEC; ++q) v[q] = 0.0f;
    }
#pragma unroll
    for (int q = 0; q < VEC; ++q) tile[rr][l + q] = v[q];
  }
  __syncthreads();
  for (int cc = tid / LPR; cc < 64; cc += RPP) {
    const int c = c0 + cc;
    if (c < C && r0 + l < Rpad) {
      u32x4_t o;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (sizeof(T) == 2)
          o[q] = uint32_t(f32_to_bf16(tile[l + 2 * q][cc])) |
                 (uint32_t(f32_to_bf16(tile[l + 2 * q + 1][cc])) << 16);
        else
          o[q] = __float_as_uint(tile[l + q][cc]);
      }
      *reinterpret_cast<u32x4_t*>(out + int64_t(c) * ldo + r0 + l) = o;
    }
  }
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * blockDim.x)
    p[i] = v;
}

// ------------------------------------------------------------------ host side

static inline int64_t rup(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Tile group of a GEMM (tile_coords), measured back to back on the two hidden sizes of the
// workloads: the logits GEMM takes 32 at K = d = 3584 (8 and 16 lose 5% and 2.5% there, 64 is
// level) and 16 at d = 1536 (+5% on that GEMM against 32; 8, 12, 20, 24 and 64 are slower
// too); dhidden 4 when d spans 14 column blocks (2, 8 and 16 lose ~1.5%) and 8 when it spans 6
// (+2% on the backward launch at d = 1536); the dW tiles 4 at both (2 and 8 lose).
static int tile_group(int mode, int32_t K, int32_t nnb) {
  if (mode == MODE_FWD) return K <= 2048 ? 16 : 32;
  if (mode == MODE_DH) return nnb <= 8 ? 8 : 4;
  return 4;
}

template <typename T, int MODE>
static int launch_gemm(GemmParams p, int kind, double flops, hipStream_t stream) {
  p.nmb = int((p.M + kBM - 1) / kBM);
  p.nnb = int((p.N + kBN - 1) / kBN);
  p.group = tile_group(MODE, p.K, p.nnb);
  const int64_t nblk = int64_t(p.nmb) * p.nnb;
  if (nblk == 0) return FASTRL_OK;
  FR_CHECK_ARG(sizeof(T) != 2 || MODE != MODE_DW ||
                   (p.K % 64 == 0 && p.lda < (int64_t(1) << 23) && p.ldb < (int64_t(1) << 23)),
               FASTRL_ERR_UNSUPPORTED,
               "dW GEMM: K must be a multiple of 64 and leading dimensions below 2^23");
  // transposed dW: whole 64-k tiles, whole 256-column tiles of the K-major E, 16-byte dW rows
  FR_CHECK_ARG(MODE != MODE_DWT || (p.K % 64 == 0 && p.ldb >= int64_t(p.nnb) * kBN &&
                                    p.ldb % 8 == 0 && p.d % 4 == 0 && p.M == p.d),
               FASTRL_ERR_UNSUPPORTED, "transposed dW GEMM: unsupported shape");
  ProfScope prof(kind, stream, flops);
  hipLaunchKernelGGL((lm_gemm_kernel<T, MODE>), dim3(unsigned(nblk)), dim3(Geo<T, MODE>::THREADS), 0,
                     stream, p);
  FR_LAUNCHED();
  return FASTRL_OK;
}

// dhidden (q, MODE_DH) and transposed dW (r, MODE_DWT) of one bf16 slab in one launch
static int launch_bwd(GemmParams q, GemmParams r, double flops, hipStream_t stream) {
  q.nmb = int((q.M + kBM - 1) / kBM);
  q.nnb = int((q.N + kBN - 1) / kBN);
  r.nmb = int((r.M + kBM - 1) / kBM);
  r.nnb = int((r.N + kBN - 1) / kBN);
  q.group = tile_group(MODE_DH, q.K, q.nnb);
  r.group = tile_group(MODE_DWT, r.K, r.nnb);
  const int64_t nh = int64_t(q.nmb) * q.nnb, nw = int64_t(r.nmb) * r.nnb;
  if (nh + nw == 0) return FASTRL_OK;
  FR_CHECK_ARG(nh + nw < (int64_t(1) << 31), FASTRL_ERR_UNSUPPORTED, "backward GEMMs: grid too large");
  FR_CHECK_ARG(r.K % 64 == 0 && r.ldb >= int64_t(r.nnb) * kBN && r.ldb % 8 == 0 && r.d % 4 == 0 &&
                   r.M == r.d,
               FASTRL_ERR_UNSUPPORTED, "transposed dW GEMM: unsupported shape");
  ProfScope prof(FASTRL_K_BACKWARD, stream, flops);
  hipLaunchKernelGGL(lm_bwd_kernel, dim3(unsigned(nh + nw)), dim3(512), 0, stream, q, r);
  FR_LAUNCHED();
  return FASTRL_OK;
}

// the second evaluation of marked token blocks (store_e == 2): bf16 through lm_redo_kernel
template <typename T>
static int launch_redo(GemmParams p, hipStream_t stream) {
  p.store_e = 2;
  if constexpr (sizeof(T) != 2) return launch_gemm<T, MODE_FWD>(p, -1, 0.0, stream);
  p.nmb = int((p.M + kBM - 1) / kBM);
  p.nnb = int((p.N + kBN - 1) / kBN);
  p.group = tile_group(MODE_FWD, p.K, p.nnb);
  const int64_t nblk = int64_t(p.nmb) * p.nnb;
  if (nblk == 0) return FASTRL_OK;
  hipLaunchKernelGGL(lm_redo_kernel, dim3(unsigned(std::min<int64_t>(nblk, 256))), dim3(512), 0,
                     stream, p);
  FR_LAUNCHED();
  return FASTRL_OK;
}

#define FR_TRY(x)                 \
  do {                            \
    int rc_ = (x);                \
    if (rc_ != FASTRL_OK) return rc_; \
  } while (0)

static inline unsigned nb1d(int64_t n, int b) { return unsigned((n + b - 1) / b); }

// ---------------------------------------------------------------- token log-prob only
constexpr int64_t kLogprobChunk = 65536;

struct LogprobWs {
  float *pmax, *psum, *zlab;
  int32_t* yslab;
};

// tokens per chunk for T tokens when at most `chunk` fit (a multiple of 256)
static int64_t logprob_chunk(int64_t T, int64_t chunk) {
  return rup(std::min<int64_t>(std::max<int64_t>(T, 1), chunk), 256);
}

static size_t carve_logprob(Carver& c, LogprobWs& w, int64_t ch, int32_t V) {
  const int64_t nmb = (V + kBM - 1) / kBM;
  w.pmax = c.take<float>(size_t(nmb * ch));
  w.psum = c.take<float>(size_t(nmb * ch));
  w.zlab = c.take<float>(size_t(ch));
  w.yslab = c.take<int32_t>(size_t(ch));
  return c.size();
}

size_t token_logprob_workspace(int64_t T, int32_t d, int32_t V, int32_t dtype) {
  (void)d;
  (void)dtype;
  Carver c(nullptr);
  LogprobWs w;
  return carve_logprob(c, w, logprob_chunk(T, kLogprobChunk), V);
}

// Chunks of at most `chunk` tokens through the logits GEMM (partials only) and the merge;
// every token's result depends on its own logits alone, so the chunking changes nothing.
// prof: record the GEMM launches in the kernel-timing recorder.
template <typename T>
static int token_logprob_impl(const void* hidden, const int32_t* row_index, const void* W,
                              int64_t Tn, int32_t d, int32_t V, const int32_t* token_ids,
                              float* logp, float* lse, int32_t* status, void* ws,
                              int64_t chunk, bool prof, hipStream_t stream) {
  Carver c(ws);
  LogprobWs w;
  const int64_t ch = logprob_chunk(Tn, chunk);
  carve_logprob(c, w, ch, V);
  for (int64_t t0 = 0; t0 < Tn; t0 += ch) {
    const int32_t Tc = int32_t(std::min<int64_t>(ch, Tn - t0));
    hipLaunchKernelGGL(slab_prep_kernel, dim3(nb1d(Tc, 256)), dim3(256), 0, stream, token_ids,
                       row_index, t0, Tc, V, w.yslab, (float*)nullptr, status);
    FR_LAUNCHED();
    GemmParams p{};
    p.A = W; p.lda = d; p.M = V;
    p.B = hidden; p.ldb = d; p.N = Tc; p.b_rows = row_index; p.b_row_base = t0;
    p.K = d;
    p.pmax = w.pmax; p.psum = w.psum; p.ldp = ch; p.zlab = w.zlab; p.yslab = w.yslab;
    p.Vreal = V; p.store_e = 0; p.status = status;
    FR_TRY((launch_gemm<T, MODE_FWD>(p, prof ? FASTRL_K_LOGITS_FWD : -1,
                                     2.0 * V * double(Tc) * d, stream)));
    const int32_t nmb = (V + kBM - 1) / kBM;
    hipLaunchKernelGGL(merge_kernel, dim3(nb1d(Tc, 64)), dim3(256), 0, stream, w.pmax, w.psum,
                       (const float*)nullptr, ch, nmb, w.zlab, w.yslab, Tc, 0, 0,
                       lse ? lse + t0 : (float*)nullptr, logp + t0, (float*)nullptr,
                       (float*)nullptr, (int32_t*)nullptr, (int32_t*)nullptr,
                       (int32_t*)nullptr, 0);
    FR_LAUNCHED();
  }
  return FASTRL_OK;
}

int run_token_logprob(const void* hidden, const int32_t* row_index, const void* W,
                      int32_t dtype, int64_t T, int32_t d, int32_t V,
                      const int32_t* token_ids, float* logp, float* lse, int32_t* status,
                      void* ws, hipStream_t stream) {
  if (dtype == FASTRL_BF16)
    return token_logprob_impl<uint16_t>(hidden, row_index, W, T, d, V, token_ids, logp, lse,
                                        status, ws, kLogprobChunk, true, stream);
  return token_logprob_impl<float>(hidden, row_index, W, T, d, V, token_ids, logp, lse, status,
                                   ws, kLogprobChunk, true, stream);
}

// ---- the allocation-free variant: its scratch is a fixed device array --------------------
// kNoAllocScratchBytes of device memory per GPU, held from the library's first use on that
// GPU until the process ends.  In host code `scratch` names a host-side stand-in, not the
// device copy: its device address is fetched once per device (hipGetSymbolAddress, with that
// device current) and only that address reaches kernels.  Every call on a GPU shares that
// GPU's array, so calls that overlap on one GPU (two streams, two threads) race.  Nothing in
// it has to start at zero: each chunk writes every partial, label and logit it reads.
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxScratchDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_dev[kMaxScratchDevices] = {};

size_t token_logprob_noalloc_scratch_bytes() { return kNoAllocScratchBytes; }

// the most tokens per chunk (a multiple of 256) whose partials fit in the scratch; 0 if not
// even 256 do
int64_t token_logprob_noalloc_chunk(int32_t V) {
  int64_t lo = 0;
  for (int64_t ch = 256; ch <= kLogprobChunk; ch += 256) {
    Carver c(nullptr);
    LogprobWs w;
    if (carve_logprob(c, w, ch, V) > kNoAllocScratchBytes) break;
    lo = ch;
  }
  return lo;
}

int run_token_logprob_noalloc(const void* hidden, const int32_t* row_index, const void* W,
                              int32_t dtype, int64_t T, int32_t d, int32_t V,
                              const int32_t* token_ids, float* logp, float* lse,
                              int32_t* status, hipStream_t stream) {
  const int64_t chunk = token_logprob_noalloc_chunk(V);
  FR_CHECK_ARG(chunk >= 256, FASTRL_ERR_SHAPE,
               "fastrl_token_logprob_noalloc: V = " + std::to_string(V) +
                   " needs more than the fixed scratch of " +
                   std::to_string(kNoAllocScratchBytes >> 20) + " MiB for 256 tokens");
  int dev = -1;
  FR_HIP(hipGetDevice(&dev));
  FR_CHECK_ARG(dev >= 0 && dev < kMaxScratchDevices, FASTRL_ERR_UNSUPPORTED,
               "fastrl_token_logprob_noalloc: device ordinal out of range");
  if (stream) {
    int sdev = -1;
    FR_HIP(hipStreamGetDevice(stream, &sdev));
    FR_CHECK_ARG(sdev == dev, FASTRL_ERR_VALUE,
                 "fastrl_token_logprob_noalloc: the stream belongs to another device than the "
                 "current one");
  }
  void* ptr = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
      void* p = nullptr;
      FR_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
      FR_CHECK_ARG(p != nullptr, FASTRL_ERR_HIP,
                   "fastrl_token_logprob_noalloc: no device address for the scratch array");
      g_scratch_dev[dev] = p;
    }
    ptr = g_scratch_dev[dev];
  }
  if (T == 0) return FASTRL_OK;
  if (dtype == FASTRL_BF16)
    return token_logprob_impl<uint16_t>(hidden, row_index, W, T, d, V, token_ids, logp, lse,
                                        status, ptr, chunk, false, stream);
  return token_logprob_impl<float>(hidden, row_index, W, T, d, V, token_ids, logp, lse, status,
                                   ptr, chunk, false, stream);
}

// ---------------------------------------------------------------- loss forward/backward
// Default slab: 32768 tokens whatever T is, so the exp-logit buffer [slab, V_pad] is bounded
// (10 GB in bf16 at V = 152064) and no [T, V] array exists for any T; a caller picks another
// bound with slab_tokens.
constexpr int64_t kDefaultSlabTokens = 32768;

struct SlabPlan {
  std::vector<int32_t> seq_begin;  // first sequence of each slab; back() == S
  int64_t tc_max = 0;
};

// Whole sequences per slab.  Each slab takes an even share of what is left, counted afresh
// after every slab (ceil(remaining / cap) slabs to go, so the shares stay close to cap): it
// ends at the sequence boundary closest to that share, never past 1.25 cap unless a single
// sequence is longer, so every slab holds at most max(1.25 cap, longest sequence) tokens.
// A slab holds at least one token while any are left (empty sequences join the slab of
// their neighbours); only T == 0 gives a slab without tokens.
static SlabPlan plan_slabs(const int64_t* off, int32_t S, int64_t cap) {
  SlabPlan pl;
  const int64_t hard = cap + cap / 4;
  int32_t i = 0;
  while (i < S) {
    pl.seq_begin.push_back(i);
    const int64_t start = off[i];
    const int64_t rem = off[S] - start;
    const int64_t left = std::max<int64_t>(1, (rem + cap - 1) / cap);
    int32_t best = S;
    if (left > 1) {
      const int64_t target = (rem + left - 1) / left;
      best = i + 1;
      while (best < S && off[best] == start) ++best;  // at least one token
      for (int32_t j = best + 1; j <= S && off[j] - start <= hard; ++j)
        if (std::llabs(off[j] - start - target) < std::llabs(off[best] - start - target)) best = j;
      while (best < S && off[best + 1] == off[best]) ++best;  // trailing empty sequences
    }
    pl.tc_max = std::max<int64_t>(pl.tc_max, off[best] - start);
    i = best;
  }
  pl.seq_begin.push_back(S);
  return pl;
}

struct LossWs {
  void *WT, *E1, *Bd;
  float *pmax, *psum, *psz, *ent, *zlab, *shift, *cslab, *lse, *logp;
  int32_t *yslab, *redo_blk, *redo_count, *seq_clip;
  double* seq_loss;
};

static size_t carve_loss(Carver& c, LossWs& w, const fastrl_loss_args& a, int64_t tc_max) {
  const int esz = a.dtype == FASTRL_BF16 ? 2 : 4;
  const int64_t Vpad = rup(a.V, kBM);
  const int64_t tcp = rup(std::max<int64_t>(tc_max, 1), kBN);
  const int64_t nmb = Vpad / kBM;
  const bool dh = a.dhidden != nullptr, dw = a.dW != nullptr;
  w.WT = dh ? c.take<char>(size_t(a.d) * Vpad * esz) : nullptr;
  w.E1 = (dh || dw) ? c.take<char>(size_t(tcp) * Vpad * esz) : nullptr;
  w.Bd = dw ? c.take<char>(size_t(a.d) * tcp * esz) : nullptr;
  w.pmax = c.take<float>(size_t(nmb * tcp));
  w.psum = c.take<float>(size_t(nmb * tcp));
  const bool ent = a.entropy != nullptr || a.entropy_sum != nullptr;
  w.psz = ent ? c.take<float>(size_t(nmb * tcp)) : nullptr;
  w.ent = a.entropy ? a.entropy
                    : (a.entropy_sum ? c.take<float>(size_t(std::max<int64_t>(a.T, 1))) : nullptr);
  w.zlab = c.take<float>(size_t(tcp));
  w.shift = c.take<float>(size_t(tcp));
  w.cslab = c.take<float>(size_t(tcp));
  w.yslab = c.take<int32_t>(size_t(tcp));
  w.redo_blk = c.take<int32_t>(size_t(tcp / kBN + 1));  // + the slab's any-marked flag
  w.redo_count = c.take<int32_t>(1);
  w.lse = a.lse ? a.lse : c.take<float>(size_t(std::max<int64_t>(a.T, 1)));
  w.logp = a.logp ? a.logp : c.take<float>(size_t(std::max<int64_t>(a.T, 1)));
  w.seq_loss = c.take<double>(size_t(std::max(a.S, 1)));
  w.seq_clip = c.take<int32_t>(size_t(std::max(a.S, 1)));
  return c.size();
}

static int64_t slab_cap(const fastrl_loss_args& a) {
  return a.slab_tokens > 0 ? a.slab_tokens : kDefaultSlabTokens;
}

int policy_loss_slab_plan(const fastrl_loss_args& a, int32_t* seq_begin, int32_t capacity,
                          int64_t* tc_max) {
  SlabPlan pl = plan_slabs(a.seq_off_host, a.S, slab_cap(a));
  const int32_t n = int32_t(pl.seq_begin.size()) - 1;
  if (tc_max) *tc_max = pl.tc_max;
  if (seq_begin && capacity > n)
    for (int32_t k = 0; k <= n; ++k) seq_begin[k] = pl.seq_begin[k];
  return n;
}

size_t policy_loss_workspace(const fastrl_loss_args& a) {
  SlabPlan pl = plan_slabs(a.seq_off_host, a.S, slab_cap(a));
  Carver c(nullptr);
  LossWs w;
  return carve_loss(c, w, a, pl.tc_max);
}

template <typename T>
static int policy_loss_impl(const fastrl_loss_args& a, hipStream_t stream) {
  SlabPlan pl = plan_slabs(a.seq_off_host, a.S, slab_cap(a));
  Carver c(a.ws);
  LossWs w;
  carve_loss(c, w, a, pl.tc_max);
  const int64_t Vpad = rup(a.V, kBM);
  const int64_t tcp = rup(std::max<int64_t>(pl.tc_max, 1), kBN);
  const int32_t nmb = int32_t(Vpad / kBM);
  const bool dh = a.dhidden != nullptr, dw = a.dW != nullptr;
  const int32_t d = a.d, V = a.V;

  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(64), 0, stream, w.redo_count, int64_t(1), 0);
  FR_LAUNCHED();
  // no token at all (S == 0, or only empty sequences): no GEMM writes dW
  if (dw && !a.dW_accumulate && a.T == 0) {
    hipLaunchKernelGGL(fill_i32_kernel, dim3(1024), dim3(256), 0, stream,
                       reinterpret_cast<int32_t*>(a.dW), int64_t(V) * d, 0);
    FR_LAUNCHED();
  }
  if (dh && a.S > 0) {
    dim3 g(nb1d(d, 64), unsigned(Vpad / 64));
    hipLaunchKernelGGL((transpose_scale_kernel<T>), g, dim3(256), 0, stream,
                       static_cast<const T*>(a.W), (const int32_t*)nullptr, int64_t(0), V,
                       int32_t(Vpad), d, (const float*)nullptr, static_cast<T*>(w.WT), Vpad);
    FR_LAUNCHED();
  }
  const size_t nslab = pl.seq_begin.size() - 1;
  bool dw_written = false;  // a slab's dW GEMM has overwritten dW
  for (size_t si = 0; si < nslab; ++si) {
    const int32_t s0 = pl.seq_begin[si], s1 = pl.seq_begin[si + 1];
    const int64_t t0 = a.seq_off_host[s0];
    const int32_t Tc = int32_t(a.seq_off_host[s1] - t0);
    if (Tc == 0) {  // only empty sequences (T == 0): their loss terms and clip counts are 0
      hipLaunchKernelGGL(loss_kernel, dim3(unsigned(s1 - s0)), dim3(256), 0, stream, w.logp,
                         w.lse, a.old_logp, a.ref_logp, a.row_index, a.seq_off, a.adv,
                         a.seq_index, a.S, a.T, s0, t0, a.algo, a.norm, a.eps_low, a.eps_high,
                         a.beta, w.shift, w.cslab, w.seq_loss, w.seq_clip, a.status,
                         a.seq_index ? INT32_MAX : a.S, (void*)nullptr, int64_t(0), 0,
                         (const int32_t*)nullptr);
      FR_LAUNCHED();
      continue;
    }
    const int64_t Tr = rup(Tc, kBN);
    const int32_t nnb = int32_t(Tr / kBN);
    hipLaunchKernelGGL(slab_prep_kernel, dim3(nb1d(Tc, 256)), dim3(256), 0, stream,
                       a.token_ids, a.row_index, t0, Tc, V, w.yslab, w.shift, a.status);
    FR_LAUNCHED();
    hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(256), 0, stream, w.redo_blk,
                       int64_t(nnb) + 1, 0);
    FR_LAUNCHED();
    GemmParams p{};
    p.A = a.W; p.lda = d; p.M = V;
    p.B = a.hidden; p.ldb = d; p.N = Tc; p.b_rows = a.row_index; p.b_row_base = t0;
    p.K = d;
    p.pmax = w.pmax; p.psum = w.psum; p.psz = w.psz; p.ldp = tcp; p.zlab = w.zlab;
    p.yslab = w.yslab; p.shift = w.shift; p.E1 = w.E1; p.ldE1 = Vpad;
    p.Vreal = V; p.store_e = (dh || dw) ? 1 : 0; p.status = a.status;
    p.redo_blk = w.redo_blk;
    p.redo_any = w.redo_blk + nnb;
    const double f_fwd = 2.0 * double(V) * Tc * d;
    FR_TRY((launch_gemm<T, MODE_FWD>(p, FASTRL_K_LOGITS_FWD, f_fwd, stream)));
    const bool store = dh || dw;
    hipLaunchKernelGGL(merge_kernel, dim3(nb1d(Tc, 64)), dim3(256), 0, stream,
                       w.pmax, w.psum, w.psz, tcp, nmb, w.zlab, w.yslab, Tc, store ? 1 : 0,
                       store ? 1 : 0, w.lse + t0, w.logp + t0, w.ent ? w.ent + t0 : nullptr,
                       store ? w.shift : (float*)nullptr, w.redo_blk, w.redo_count,
                       w.redo_blk + nnb, 0);
    FR_LAUNCHED();
    if (store) {
      // token blocks holding a row that needs a shift: evaluate again, then merge again (both
      // return at once on the device when no row was marked)
      FR_TRY(launch_redo<T>(p, stream));
      hipLaunchKernelGGL(merge_kernel, dim3(nb1d(Tc, 64)), dim3(256), 0, stream,
                         w.pmax, w.psum, w.psz, tcp, nmb, w.zlab, w.yslab, Tc, 1, 0, w.lse + t0,
                         w.logp + t0, w.ent ? w.ent + t0 : nullptr, w.shift, w.redo_blk,
                         w.redo_count, w.redo_blk + nnb, 1);
      FR_LAUNCHED();
    }
    hipLaunchKernelGGL(loss_kernel, dim3(unsigned(s1 - s0)), dim3(256), 0, stream, w.logp,
                       w.lse, a.old_logp, a.ref_logp, a.row_index, a.seq_off, a.adv,
                       a.seq_index, a.S, a.T, s0, t0, a.algo, a.norm, a.eps_low, a.eps_high,
                       a.beta, w.shift, w.cslab, w.seq_loss, w.seq_clip, a.status,
                       a.seq_index ? INT32_MAX : a.S, store ? w.E1 : nullptr, Vpad,
                       sizeof(T) == 2 ? 1 : 0, w.yslab);
    FR_LAUNCHED();
    GemmParams q{};  // dhidden: C = E W^T (rows = tokens, cols = d, K = padded vocabulary)
    if (dh) {
      q.A = w.E1; q.lda = Vpad; q.M = Tc;
      q.B = w.WT; q.ldb = Vpad; q.N = d;
      q.K = int32_t(Vpad);
      q.dH = a.dhidden_dtype == FASTRL_BF16
                 ? (void*)(static_cast<uint16_t*>(a.dhidden) + t0 * d)
                 : (void*)(static_cast<float*>(a.dhidden) + t0 * d);
      q.dH_bf16 = a.dhidden_dtype == FASTRL_BF16;
      q.cslab = w.cslab; q.d = d;
      q.status = a.status;
    }
    // bf16 with both gradients: the two GEMMs run as one launch (after dW's inputs are ready)
    const bool fused = dh && dw && sizeof(T) == 2;
    if (dh && !fused)
      FR_TRY((launch_gemm<T, MODE_DH>(q, FASTRL_K_DHIDDEN, 2.0 * double(Tc) * d * V, stream)));
    if (dw) {
      dim3 g(nb1d(d, 64), unsigned(Tr / 64));
      hipLaunchKernelGGL((transpose_scale_kernel<T>), g, dim3(256), 0, stream,
                         static_cast<const T*>(a.hidden), a.row_index, t0, Tc, int32_t(Tr), d,
                         w.cslab, static_cast<T*>(w.Bd), tcp);
      FR_LAUNCHED();
      GemmParams r{};
      r.K = int32_t(Tr);
      r.dW = a.dW; r.dW_acc = (dw_written || a.dW_accumulate) ? 1 : 0;
      r.d = d;
      r.status = a.status;
      if constexpr (sizeof(T) == 2) {  // dW^T = Bd E: A = Bd, B = E1 read K-major
        r.A = w.Bd; r.lda = tcp; r.M = d;
        r.B = w.E1; r.ldb = Vpad; r.N = V;
        if (fused)
          FR_TRY(launch_bwd(q, r, 4.0 * double(V) * d * Tc, stream));
        else
          FR_TRY((launch_gemm<T, MODE_DWT>(r, FASTRL_K_DW, 2.0 * double(V) * d * Tc, stream)));
      } else {  // dW = E^T Bd^T: A = E1 read K-major (A[v][t] = E1[t][v]), B = Bd
        r.A = w.E1; r.lda = Vpad; r.M = V;
        r.B = w.Bd; r.ldb = tcp; r.N = d;
        FR_TRY((launch_gemm<T, MODE_DW>(r, FASTRL_K_DW, 2.0 * double(V) * d * Tc, stream)));
      }
      dw_written = true;
    }
  }
  hipLaunchKernelGGL(loss_final_kernel, dim3(1), dim3(256), 0, stream, w.seq_loss, w.seq_clip,
                     a.S, w.redo_count, a.loss, a.stats);
  FR_LAUNCHED();
  if (a.entropy_sum) {
    hipLaunchKernelGGL(sum_f32_kernel, dim3(1), dim3(256), 0, stream, w.ent, a.T,
                       a.entropy_sum);
    FR_LAUNCHED();
  }
  return FASTRL_OK;
}

int run_policy_loss(const fastrl_loss_args& a, hipStream_t stream) {
  if (a.dtype == FASTRL_BF16) return policy_loss_impl<uint16_t>(a, stream);
  return policy_loss_impl<float>(a, stream);
}

}  // namespace fastrl
