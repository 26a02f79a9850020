// Prefill product on the Tiled-CBC arrays (Sec. 4.3): Y = X W_sp^T for N
// tokens with static pruning only (no activation test), on gfx950's matrix
// cores. The weights stay in the decode format -- the same handle serves
// both phases -- and are expanded tile by tile into a dense operand in LDS
// (the paper's layout-alignment stage), then multiplied with
// v_mfma_f32_32x32x16_f16 (fp16 operands, fp32 accumulation).
//
// A workgroup owns one 256-row stripe x 128 tokens and walks the stripe in
// k-steps of 16 columns. Expansion of a k-step: lane i of bitmap word v of
// a column takes row 64 v + i; its value sits at the word's masked popcount
// below bit i plus the popcounts of the column's earlier words (HAD-SMBD,
// Sec. 4.2.1), or is 0 where the bit is clear; the tile is row-major, 16
// fp16 per row, rows padded to 40 bytes so that the MFMA operand reads of
// 32 consecutive rows spread over the banks.
//
// Two forms:
//   * spmm_kernel, any tile_k >= 16 and any width: four waves, each expands
//     four columns and multiplies the stripe's eight 32-row blocks with its
//     32 tokens; operands fetched one step ahead into registers;
//   * spmm_ws_kernel, 256 x 16 GTiles and a width that is a multiple of 8:
//     warp-specialized, DMA ring, split-K over the GTiles when the grid is
//     small (described at the kernel).

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "internal.h"

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));

constexpr int kTM = 256;                       // rows of a stripe (four bitmap words per column)
constexpr int kKStep = 16;                     // columns per k-step (the MFMA's k)
constexpr int kWaves = 4;
constexpr int kTokPerWave = 32;
constexpr int kBN = kWaves * kTokPerWave;      // tokens per workgroup
constexpr int kRowBytes = 40;                  // a dense-tile row: 16 fp16 + 8 bytes of padding
constexpr int kTileBytes = kTM * kRowBytes;
constexpr int kBlocks = kTM / 32;              // 32-row MFMA blocks of a stripe

struct SpmmArgs {
  const uint32_t* tile_offset;
  const uint32_t* col_info;
  const uint64_t* bitmap;
  const uint16_t* values;
  const uint16_t* x;  // [n_tokens][cols]
  uint16_t* y;        // [n_tokens][rows]
  long long n_tokens;
  int rows, cols;
  int tk_log2;        // tile_k = 1 << tk_log2 >= 16
  int n_colblocks;
  int steps;          // k-steps over the padded width: n_colblocks * tile_k / 16
  int x_vec;          // cols % 8 == 0: X rows are read 16 bytes at a time
  int y_vec;          // rows % 4 == 0: Y rows are written 8 bytes at a time
};

__device__ __forceinline__ uint32_t mbcnt64(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

template <class T>
using const_ptr = const __attribute__((address_space(4))) T*;

// The plain form. What one wave fetches for one k-step: its four columns'
// values (one per lane and bitmap word, 0 where the bit is clear) and its B
// operand.
struct StepData {
  uint2 v[4];  // [word]: the four columns' fp16 bits, two per dword
  half8 b;
};

__global__ __launch_bounds__(256) void spmm_kernel(SpmmArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char tile[2][kTileBytes];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = blockIdx.x;  // stripe
  const long long n_wave = (long long)blockIdx.y * kBN + (long long)wave * kTokPerWave;
  const int tk = 1 << a.tk_log2;
  const int khalf = (lane >> 5) * 8;
  // this lane's token for the B operand (tokens past the end re-read the
  // last one; their outputs are not written)
  const long long tok = n_wave + (lane & 31) < a.n_tokens ? n_wave + (lane & 31) : a.n_tokens - 1;
  const uint16_t* const xrow = a.x + tok * (long long)a.cols;
  const const_ptr<uint32_t> ci_s = (const_ptr<uint32_t>)a.col_info;
  const const_ptr<uint32_t> to_s = (const_ptr<uint32_t>)a.tile_offset;
  const const_ptr<uint64_t> bm_s = (const_ptr<uint64_t>)a.bitmap;

  auto fetch = [&](int s, StepData& d) __attribute__((always_inline)) {
    const int k0 = s * kKStep;
    const int c = k0 >> a.tk_log2;
    const int g = r * a.n_colblocks + c;
    const uint32_t col0 = (uint32_t)g * (uint32_t)tk + (uint32_t)(k0 - (c << a.tk_log2)) + 4u * (uint32_t)wave;
    const uint32_t to = to_s[g];
    uint32_t h[4][4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const uint32_t ci = ci_s[col0 + jj];
      uint32_t base = to + (ci >> 16);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const uint64_t word = bm_s[(size_t)(col0 + jj) * 4 + v];
        h[v][jj] = 0;
        if ((word >> lane) & 1) h[v][jj] = a.values[base + mbcnt64(word)];
        base += (uint32_t)__builtin_popcountll(word);
      }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) d.v[v] = make_uint2(h[v][0] | (h[v][1] << 16), h[v][2] | (h[v][3] << 16));
    // B operand: X[tok][k0 + khalf .. + 8], zero past the last column
    const int kb = k0 + khalf;
    if (a.x_vec) {
      if (kb < a.cols) {
        d.b = *reinterpret_cast<const half8*>(xrow + kb);
      } else {
        d.b = half8{0, 0, 0, 0, 0, 0, 0, 0};
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint16_t hx = kb + e < a.cols ? xrow[kb + e] : (uint16_t)0;
        d.b[e] = __builtin_bit_cast(_Float16, hx);
      }
    }
  };

  float16v acc[kBlocks];
#pragma unroll
  for (int i = 0; i < kBlocks; ++i) acc[i] = float16v{};

  StepData cur, nxt;
  fetch(0, cur);
  for (int s = 0; s < a.steps; ++s) {
    unsigned char* t = tile[s & 1];
    // 1. this wave's four columns into rows 64v + lane of the dense tile
#pragma unroll
    for (int v = 0; v < 4; ++v) *reinterpret_cast<uint2*>(t + (64 * v + lane) * kRowBytes + 8 * wave) = cur.v[v];
    __syncthreads();
    if (s + 1 < a.steps) fetch(s + 1, nxt);
    // 2. the stripe's eight 32-row blocks times this wave's 32 tokens
    const half8 b = cur.b;
#pragma unroll
    for (int i = 0; i < kBlocks; ++i) {
      const unsigned char* p = t + (32 * i + (lane & 31)) * kRowBytes + 2 * khalf;
      const uint2 lo = *reinterpret_cast<const uint2*>(p);
      const uint2 hi = *reinterpret_cast<const uint2*>(p + 8);
      const half8 av = __builtin_bit_cast(half8, make_uint4(lo.x, lo.y, hi.x, hi.y));
      acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, b, acc[i], 0, 0, 0);
    }
    cur = nxt;
  }

  // 3. accumulator register e of block i holds row 32 i + 8 (e / 4) +
  // 4 (lane / 32) + e % 4 and token lane % 32: four consecutive rows per
  // group of four registers, rounded once to fp16
  const long long n = n_wave + (lane & 31);
  if (n >= a.n_tokens) return;
  uint16_t* const yrow = a.y + n * (long long)a.rows;
#pragma unroll
  for (int i = 0; i < kBlocks; ++i) {
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const int m = r * kTM + 32 * i + 8 * grp + 4 * (lane >> 5);
      uint16_t h[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = __half_as_ushort(__float2half_rn(acc[i][4 * grp + e]));
      if (a.y_vec && m + 3 < a.rows) {
        *reinterpret_cast<uint2*>(yrow + m) = make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (m + e < a.rows) yrow[m + e] = h[e];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Helpers of the pipelined form below.

constexpr int kValBytes = kTM * kKStep * 2;    // a dense GTile's worth of values
constexpr int kXBytes = kBN * kKStep * 2;      // 128 tokens x 16 columns

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// Global -> LDS DMA (lane l's bytes land at lds + 16 l, or + 4 l). Issued as
// assembly so that the compiler does not order LDS reads of other ring
// slots behind every outstanding load; the waits are explicit. The compiler
// does not look inside assembly for hazards: a vector memory instruction
// needs 5 wait states after a VALU write of an SGPR it reads, hence s_nop 4.
__device__ __forceinline__ void dma16(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(lds) : "memory");
}
__device__ __forceinline__ void dma4(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_nop 4\n\tglobal_load_lds_dword %0, %1" ::"v"(off), "s"(base), "{m0}"(lds) : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// ---------------------------------------------------------------------------
// Warp-specialized form, for 256 x 16 GTiles and a width that is a
// multiple of 8 (every Llama shape): each k-step is one GTile, and what a
// step reads from memory -- the GTile's padded values (one contiguous run)
// and the 128 x 16 block of X -- is copied into a ring of LDS slots by
// global->LDS DMA several steps ahead. Sixteen waves: waves 0-7 multiply, waves
// 8-15 expand. A wave issues in order and waits while the matrix core is
// busy with its previous MFMA, so a wave that did both would serialize
// them; with the roles in different waves every SIMD holds two multiplying
// and two expanding waves, and the expansion of step s + 1 runs while the
// MFMAs of step s do. One barrier per step (one GTile).
//   * multiplying wave m: rows 64 (m & 3) .., tokens 64 (m >> 2) .. of the
//     256 x 128 output tile (four 32 x 32 blocks, A and B each read once);
//     it also issues the step's DMA: one 16-byte load of values (8 x 64
//     lanes x 16 bytes cover a dense GTile) and one of X (m < 4: 32 tokens
//     each) or of bitmap words / ColInfo (m >= 4: these only warm L2 for
//     the expanding waves' scalar loads and land in a scratch area). The
//     TileOffsets come from the LDS table: no scalar memory load, so the
//     LDS waits of these waves never wait for one;
//   * expanding wave d: columns 2d, 2d + 1 of the GTile (eight bitmap
//     words, scalar loads two steps ahead, so the loads of step s + 2 are in
//     flight while step s + 1 is expanded), values from the slot.
// A slot is refilled in the step after its X rows were read: step s
// requests step s + kWsRing - 1 into the slot of step s - 1.
//
// Split-K (blockIdx.z of k_splits): a workgroup walks GTiles [z sps, (z + 1)
// sps) of its stripe and, with more than one split, stores its fp32 sums to
// part[z][token][row]; spmm_reduce_kernel adds the splits in order.

constexpr int kWsWaves = 16;
constexpr int kWsRing = 8;
constexpr int kWsDma = 2;      // loads per step of a multiplying wave
constexpr int kToCap = 1800;   // TileOffsets of one stripe's split held in LDS
constexpr int kGBytes = kValBytes + kXBytes;  // one GTile's values and X block in a ring slot

// the lane's value where its bit of the word is set, else 0 (the word as
// the select mask of a VOP3 select: no move through vcc)
__device__ __forceinline__ uint32_t select_word(uint32_t v, uint64_t mask) {
  uint32_t r;
  asm("v_cndmask_b32_e64 %0, 0, %1, %2" : "=v"(r) : "v"(v), "s"(mask));
  return r;
}

// wait until at most kWsDma x `later` loads are in flight (later < N + 1)
template <int N>
__device__ __forceinline__ void wait_steps(int later) {
  if constexpr (N > 0) {
    if (later >= N) {
      wait_vmcnt<kWsDma * N>();
      return;
    }
    wait_steps<N - 1>(later);
  } else {
    wait_vmcnt<0>();
  }
}

struct WsArgs {
  SpmmArgs s;
  float* part;  // [k_splits][n_tokens][rows] fp32 when k_splits > 1
  int k_splits;
  int sps;      // GTiles per split
};

__global__ __launch_bounds__(kWsWaves * 64) void spmm_ws_kernel(WsArgs wa) {
  const SpmmArgs& a = wa.s;
  __shared__ __attribute__((aligned(1024))) unsigned char ring[kWsRing][kGBytes];
  __shared__ __attribute__((aligned(16))) unsigned char tile[2][kTileBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char warm[1024];
  __shared__ uint32_t toff[kToCap];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool mma = wave < 8;
  const int mw = wave & 7;  // index within the role
  const int r = blockIdx.x;
  const long long nb0 = (long long)blockIdx.y * kBN;
  const int khalf = (lane >> 5) * 8;
  const int c0 = (int)blockIdx.z * wa.sps;                 // first GTile of this split
  const int steps = min(wa.sps, a.n_colblocks - c0);       // >= 1 (the host makes every split non-empty)
  const uint32_t g0 = (uint32_t)r * (uint32_t)a.n_colblocks;
  for (int i = threadIdx.x; i <= steps; i += kWsWaves * 64) toff[i] = a.tile_offset[g0 + (uint32_t)(c0 + i)];

  // multiplying waves: the second DMA of a GTile, as (source, lane offset
  // at GTile 0, bytes per GTile, LDS offset): X into the slot, or bitmap
  // words / ColInfo into the warm-up area
  const bool x_dma = mw < 4;
  const void* d_src;
  uint32_t d_off, d_step, d_lds;
  {
    const long long left = a.n_tokens - nb0;
    const int xt = 32 * mw + (lane >> 1);
    if (x_dma) {
      d_src = a.x + nb0 * (long long)a.cols;
      d_off = (uint32_t)((xt < left ? xt : left - 1) * (long long)a.cols * 2) + 16u * (uint32_t)(lane & 1);
      d_step = 2u * kKStep;
      d_lds = (uint32_t)(kValBytes + 1024 * mw);
    } else if (mw < 6) {
      d_src = a.bitmap;
      d_off = g0 * 512u + 256u * (uint32_t)(mw - 4) + 4u * (uint32_t)lane;
      d_step = 512u;
      d_lds = lds_addr(warm) + 256u * (uint32_t)(mw - 4);
    } else {
      d_src = a.col_info;
      d_off = g0 * 64u + 4u * (uint32_t)(lane & 15);
      d_step = 64u;
      d_lds = lds_addr(warm) + 512u + 256u * (uint32_t)(mw - 6);
    }
  }
  const uint32_t q16 = 16u * (uint32_t)(mw * 64 + lane);
  __syncthreads();

  // requests step s (GTile c0 + s) into its slot
  auto issue = [&](int s) __attribute__((always_inline)) {
    const uint32_t c = (uint32_t)(c0 + s);
    const uint32_t slot = lds_addr(ring[s & (kWsRing - 1)]);
    // the GTile's values: lanes past the end re-read its last 16 bytes
    const uint32_t t0 = toff[s], t1 = toff[s + 1];
    const int span = 2 * (int)(t1 - t0) - 16;
    const uint32_t voff = 2u * t0 + min(q16, (uint32_t)max(span, 0));
    asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(a.values),
                 "{m0}"((uint32_t)__builtin_amdgcn_readfirstlane((int)(slot + 1024u * (uint32_t)mw)))
                 : "memory");
    if (x_dma) {
      // columns past the width (the last GTile of a width that is not a
      // multiple of 16): any valid 16 bytes, the B operand is cleared
      uint32_t off = d_off + c * d_step;
      if (c * kKStep + 8u * (uint32_t)(lane & 1) >= (uint32_t)a.cols) off = d_off - 16u * (uint32_t)(lane & 1);
      dma16(d_src, off, (uint32_t)__builtin_amdgcn_readfirstlane((int)(slot + d_lds)));
    } else {
      dma4(d_src, d_off + c * d_step, d_lds);
    }
  };

  // expanding waves: the two columns' words and ColInfo, by scalar loads
  struct Meta {
    uint64_t w[8];  // column 2d: words 0-3, column 2d + 1: words 4-7
    uint32_t ci[2];
  };
  const const_ptr<uint64_t> bm_s = (const_ptr<uint64_t>)a.bitmap;
  const const_ptr<uint32_t> ci_s = (const_ptr<uint32_t>)a.col_info;
  auto load_meta = [&](int s, Meta& m) __attribute__((always_inline)) {
    const uint32_t col0 = (g0 + (uint32_t)(c0 + s)) * (uint32_t)kKStep + 2u * (uint32_t)mw;
#pragma unroll
    for (int i = 0; i < 8; ++i) m.w[i] = bm_s[(size_t)col0 * 4 + i];
    m.ci[0] = ci_s[col0];
    m.ci[1] = ci_s[col0 + 1];
  };
  // column 2 d + jj, word v -> row 64 v + lane: the value at the word's
  // masked popcount below the lane plus the column's earlier words' counts
  auto decode = [&](int s, const Meta& m) __attribute__((always_inline)) {
    const uint32_t vb = lds_addr(ring[s & (kWsRing - 1)]);
    unsigned char* t = tile[s & 1];
    uint32_t hv[2][4];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      uint32_t sb = vb + 2u * (m.ci[jj] >> 16);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        hv[jj][v] = *(const __attribute__((address_space(3))) uint16_t*)(uintptr_t)(sb + 2u * mbcnt64(m.w[4 * jj + v]));
        if (v < 3) {
          const uint32_t pop = (uint32_t)__builtin_popcountll(m.w[4 * jj + v]);
          asm("s_lshl1_add_u32 %0, %1, %0" : "+s"(sb) : "s"(pop) : "scc");
        }
      }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v)
      *reinterpret_cast<uint32_t*>(t + (64 * v + lane) * kRowBytes + 4 * mw) =
          select_word(hv[0][v], m.w[v]) | (select_word(hv[1][v], m.w[4 + v]) << 16);
  };

  const int rq = mw & 3, th = mw >> 2;
  float16v acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = float16v{};
  const half8 none = half8{0, 0, 0, 0, 0, 0, 0, 0};

  // one step. Multiplying waves: MFMAs of step s, request of step
  // s + kWsRing - 1, wait for step s + 2. Expanding waves: scalar loads of
  // step s + 2 into `next`, expansion of step s + 1 from `cur`. Barrier.
  // STEADY: every one of these happens, kWsRing - 3 later steps are in
  // flight, and every column is inside the width.
  auto step = [&](int s, Meta& cur, Meta& next, auto steady) __attribute__((always_inline)) {
    constexpr bool kSteady = decltype(steady)::value;
    if (mma) {
      const unsigned char* slot = ring[s & (kWsRing - 1)];
      const unsigned char* t = tile[s & 1];
      half8 b[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        b[j] = *reinterpret_cast<const half8*>(slot + kValBytes + (64 * th + 32 * j + (lane & 31)) * 32 + 2 * khalf);
        if constexpr (!kSteady)
          if ((c0 + s) * kKStep + khalf >= a.cols) b[j] = none;
      }
      half8 av[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const unsigned char* p = t + (64 * rq + 32 * i + (lane & 31)) * kRowBytes + 2 * khalf;
        const uint2 lo = *reinterpret_cast<const uint2*>(p);
        const uint2 hi = *reinterpret_cast<const uint2*>(p + 8);
        av[i] = __builtin_bit_cast(half8, make_uint4(lo.x, lo.y, hi.x, hi.y));
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[i], b[j], acc[i][j], 0, 0, 0);
      if (kSteady || s + kWsRing - 1 < steps) issue(s + kWsRing - 1);
      if constexpr (kSteady)
        wait_vmcnt<kWsDma * (kWsRing - 3)>();
      else if (s + 2 < steps)
        wait_steps<kWsRing - 3>(min(kWsRing - 3, steps - 1 - (s + 2)));
    } else {
      if (kSteady || s + 2 < steps) load_meta(s + 2, next);
      if (kSteady || s + 1 < steps) decode(s + 1, cur);
    }
    __syncthreads();
  };

  // prologue: steps 0 .. kWsRing - 2 requested; step 0 expanded; step 1 landed
  Meta ma, mb;
  if (mma) {
    for (int s = 0; s < kWsRing - 1 && s < steps; ++s) issue(s);
    wait_steps<kWsRing - 2>(min(kWsRing - 2, steps - 1));
  } else {
    load_meta(0, ma);
    if (steps > 1) load_meta(1, mb);
  }
  __syncthreads();
  if (mma) {
    if (steps > 1) wait_steps<kWsRing - 3>(min(kWsRing - 3, steps - 2));
  } else {
    decode(0, ma);
  }
  __syncthreads();

  // step s expands s + 1 from the set loaded two steps before: step 0 uses
  // mb (step 1) and loads step 2 into ma, step 1 the other way round
  int s = 0;
  const int steady_end = steps - kWsRing;
  for (; s + 1 < steady_end; s += 2) {
    step(s, mb, ma, std::integral_constant<bool, true>{});
    step(s + 1, ma, mb, std::integral_constant<bool, true>{});
  }
  for (; s < steps; s += 2) {
    step(s, mb, ma, std::integral_constant<bool, false>{});
    if (s + 1 < steps) step(s + 1, ma, mb, std::integral_constant<bool, false>{});
  }

  if (!mma) return;
  // accumulator register e of block (i, j) holds row 32 i + 8 (e / 4) +
  // 4 (lane / 32) + e % 4 of the wave's 64 rows and token 32 j + lane % 32
  float* const part = wa.k_splits > 1 ? wa.part + (size_t)blockIdx.z * (size_t)a.n_tokens * (size_t)a.rows : nullptr;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const long long n = nb0 + 64 * th + 32 * j + (lane & 31);
    if (n >= a.n_tokens) continue;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int m = r * kTM + 64 * rq + 32 * i + 8 * grp + 4 * (lane >> 5);
        if (part) {
          float* const prow = part + n * (long long)a.rows;
          if (a.y_vec && m + 3 < a.rows) {
            *reinterpret_cast<float4*>(prow + m) = make_float4(acc[i][j][4 * grp], acc[i][j][4 * grp + 1],
                                                               acc[i][j][4 * grp + 2], acc[i][j][4 * grp + 3]);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (m + e < a.rows) prow[m + e] = acc[i][j][4 * grp + e];
          }
          continue;
        }
        uint16_t* const yrow = a.y + n * (long long)a.rows;
        uint16_t hh[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) hh[e] = __half_as_ushort(__float2half_rn(acc[i][j][4 * grp + e]));
        if (a.y_vec && m + 3 < a.rows) {
          *reinterpret_cast<uint2*>(yrow + m) =
              make_uint2(hh[0] | ((uint32_t)hh[1] << 16), hh[2] | ((uint32_t)hh[3] << 16));
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (m + e < a.rows) yrow[m + e] = hh[e];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// 256-token form of the warp-specialized kernel: the expansion of a GTile
// is an instruction stream of fixed length whatever the token count, so a
// workgroup of 256 tokens pays it once for twice the MFMA work. Twelve
// waves (three per SIMD: two multiplying, one expanding):
//   * multiplying wave m (0-7): rows 64 (m & 3) .., tokens 128 (m >> 2) ..
//     of the 256 x 256 output tile (2 x 4 blocks of 32 x 32, 128
//     accumulators); per step one 16-byte DMA of values (8 x 64 lanes x 16
//     bytes: a dense GTile) and one of X (tokens 32 m .. 32 m + 31);
//   * expanding wave d (8-11): columns 4d .. 4d + 3 (sixteen bitmap words,
//     scalar loads two steps ahead); it also warms L2 for its own scalar
//     loads (a DMA of the words it will load, into a scratch area, never
//     waited for).
// The two roles run separate loops with the same number of barriers, so
// neither role's registers are held across the other's code.

constexpr int kW256Waves = 12;
constexpr int kW256Ring = 8;
constexpr int kBN256 = 256;
constexpr int kX256Bytes = kBN256 * kKStep * 2;
constexpr int kG256Bytes = kValBytes + kX256Bytes;

__global__ __launch_bounds__(kW256Waves * 64) void spmm_ws256_kernel(WsArgs wa) {
  const SpmmArgs& a = wa.s;
  __shared__ __attribute__((aligned(1024))) unsigned char ring[kW256Ring][kG256Bytes];
  __shared__ __attribute__((aligned(16))) unsigned char tile[2][kTileBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char warm[1024];
  __shared__ uint32_t toff[kToCap];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = blockIdx.x;
  const long long nb0 = (long long)blockIdx.y * kBN256;
  const int c0 = (int)blockIdx.z * wa.sps;
  const int steps = min(wa.sps, a.n_colblocks - c0);
  const uint32_t g0 = (uint32_t)r * (uint32_t)a.n_colblocks;
  for (int i = threadIdx.x; i <= steps; i += kW256Waves * 64) toff[i] = a.tile_offset[g0 + (uint32_t)(c0 + i)];
  __syncthreads();
  constexpr int R = kW256Ring;
  const int steady_end = steps - R;

  if (wave < 8) {
    // ---- multiplying waves
    const int mw = wave;
    const int khalf = (lane >> 5) * 8;
    const int rq = mw & 3, th = mw >> 2;
    const long long left = a.n_tokens - nb0;
    const int xt = 32 * mw + (lane >> 1);
    const uint16_t* const xsrc = a.x + nb0 * (long long)a.cols;
    const uint32_t x_off = (uint32_t)((xt < left ? xt : left - 1) * (long long)a.cols * 2) + 16u * (uint32_t)(lane & 1);
    const uint32_t q16 = 16u * (uint32_t)(mw * 64 + lane);
    auto issue = [&](int s) __attribute__((always_inline)) {
      const uint32_t c = (uint32_t)(c0 + s);
      const uint32_t slot = lds_addr(ring[s & (R - 1)]);
      const uint32_t t0 = toff[s], t1 = toff[s + 1];
      const int span = 2 * (int)(t1 - t0) - 16;
      const uint32_t voff = 2u * t0 + min(q16, (uint32_t)max(span, 0));
      asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(a.values),
                   "{m0}"((uint32_t)__builtin_amdgcn_readfirstlane((int)(slot + 1024u * (uint32_t)mw)))
                   : "memory");
      uint32_t off = x_off + c * (2u * kKStep);
      if (c * kKStep + 8u * (uint32_t)(lane & 1) >= (uint32_t)a.cols) off = x_off - 16u * (uint32_t)(lane & 1);
      dma16(xsrc, off, (uint32_t)__builtin_amdgcn_readfirstlane((int)(slot + kValBytes + 1024u * (uint32_t)mw)));
    };
    float16v acc[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = float16v{};
    const half8 none = half8{0, 0, 0, 0, 0, 0, 0, 0};
    auto step = [&](int s, auto steady) __attribute__((always_inline)) {
      constexpr bool kSteady = decltype(steady)::value;
      const unsigned char* slot = ring[s & (R - 1)];
      const unsigned char* t = tile[s & 1];
      half8 av[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const unsigned char* p = t + (64 * rq + 32 * i + (lane & 31)) * kRowBytes + 2 * khalf;
        const uint2 lo = *reinterpret_cast<const uint2*>(p);
        const uint2 hi = *reinterpret_cast<const uint2*>(p + 8);
        av[i] = __builtin_bit_cast(half8, make_uint4(lo.x, lo.y, hi.x, hi.y));
      }
      const bool zero_b = !kSteady && (c0 + s) * kKStep + khalf >= a.cols;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        half8 b = *reinterpret_cast<const half8*>(slot + kValBytes + (128 * th + 32 * j + (lane & 31)) * 32 + 2 * khalf);
        if (zero_b) b = none;
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[i], b, acc[i][j], 0, 0, 0);
      }
      if (kSteady || s + R - 1 < steps) issue(s + R - 1);
      if constexpr (kSteady)
        wait_vmcnt<kWsDma * (R - 3)>();
      else if (s + 2 < steps)
        wait_steps<R - 3>(min(R - 3, steps - 1 - (s + 2)));
      __syncthreads();
    };
    for (int s = 0; s < R - 1 && s < steps; ++s) issue(s);
    wait_steps<R - 2>(min(R - 2, steps - 1));
    __syncthreads();
    if (steps > 1) wait_steps<R - 3>(min(R - 3, steps - 2));
    __syncthreads();
    int s = 0;
    for (; s < steady_end; ++s) step(s, std::integral_constant<bool, true>{});
    for (; s < steps; ++s) step(s, std::integral_constant<bool, false>{});

    float* const part = wa.k_splits > 1 ? wa.part + (size_t)blockIdx.z * (size_t)a.n_tokens * (size_t)a.rows : nullptr;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const long long n = nb0 + 128 * th + 32 * j + (lane & 31);
      if (n >= a.n_tokens) continue;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          const int m = r * kTM + 64 * rq + 32 * i + 8 * grp + 4 * (lane >> 5);
          if (part) {
            float* const prow = part + n * (long long)a.rows;
            if (a.y_vec && m + 3 < a.rows) {
              *reinterpret_cast<float4*>(prow + m) = make_float4(acc[i][j][4 * grp], acc[i][j][4 * grp + 1],
                                                                 acc[i][j][4 * grp + 2], acc[i][j][4 * grp + 3]);
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (m + e < a.rows) prow[m + e] = acc[i][j][4 * grp + e];
            }
            continue;
          }
          uint16_t* const yrow = a.y + n * (long long)a.rows;
          uint16_t hh[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) hh[e] = __half_as_ushort(__float2half_rn(acc[i][j][4 * grp + e]));
          if (a.y_vec && m + 3 < a.rows) {
            *reinterpret_cast<uint2*>(yrow + m) =
                make_uint2(hh[0] | ((uint32_t)hh[1] << 16), hh[2] | ((uint32_t)hh[3] << 16));
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (m + e < a.rows) yrow[m + e] = hh[e];
          }
        }
      }
    }
  } else {
    // ---- expanding waves
    const int d = wave - 8;
    struct Meta {
      uint64_t w[16];  // column 4d + jj: words 4 jj .. 4 jj + 3
      uint32_t ci[4];
    };
    const const_ptr<uint64_t> bm_s = (const_ptr<uint64_t>)a.bitmap;
    const const_ptr<uint32_t> ci_s = (const_ptr<uint32_t>)a.col_info;
    auto load_meta = [&](int s, Meta& m) __attribute__((always_inline)) {
      const uint32_t col0 = (g0 + (uint32_t)(c0 + s)) * (uint32_t)kKStep + 4u * (uint32_t)d;
#pragma unroll
      for (int i = 0; i < 16; ++i) m.w[i] = bm_s[(size_t)col0 * 4 + i];
#pragma unroll
      for (int i = 0; i < 4; ++i) m.ci[i] = ci_s[col0 + i];
    };
    // the words (128 bytes: two lanes of 64) and ColInfo (16 bytes) of step
    // s into L2, landing in a scratch area nobody reads
    auto warm_up = [&](int s) __attribute__((always_inline)) {
      const uint32_t col0 = (g0 + (uint32_t)(c0 + s)) * (uint32_t)kKStep + 4u * (uint32_t)d;
      dma4(a.bitmap, col0 * 32u + 4u * (uint32_t)(lane & 31), lds_addr(warm) + 256u * (uint32_t)d);
      dma4(a.col_info, col0 * 4u + 4u * (uint32_t)(lane & 3), lds_addr(warm) + 256u * (uint32_t)d);
    };
    auto decode = [&](int s, const Meta& m) __attribute__((always_inline)) {
      const uint32_t vb = lds_addr(ring[s & (R - 1)]);
      unsigned char* t = tile[s & 1];
      uint32_t hv[4][4];  // [column][word]
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        uint32_t sb = vb + 2u * (m.ci[jj] >> 16);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          hv[jj][v] = *(const __attribute__((address_space(3))) uint16_t*)(uintptr_t)(sb + 2u * mbcnt64(m.w[4 * jj + v]));
          if (v < 3) {
            const uint32_t pop = (uint32_t)__builtin_popcountll(m.w[4 * jj + v]);
            asm("s_lshl1_add_u32 %0, %1, %0" : "+s"(sb) : "s"(pop) : "scc");
          }
        }
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        uint32_t sel[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) sel[jj] = select_word(hv[jj][v], m.w[4 * jj + v]);
        *reinterpret_cast<uint2*>(t + (64 * v + lane) * kRowBytes + 8 * d) =
            make_uint2(sel[0] | (sel[1] << 16), sel[2] | (sel[3] << 16));
      }
    };
    auto step = [&](int s, Meta& cur, Meta& next, auto steady) __attribute__((always_inline)) {
      constexpr bool kSteady = decltype(steady)::value;
      if (kSteady || s + 4 < steps) warm_up(s + 4);
      if (kSteady || s + 2 < steps) load_meta(s + 2, next);
      if (kSteady || s + 1 < steps) decode(s + 1, cur);
      __syncthreads();
    };
    Meta ma, mb;
    for (int s = 0; s < 4 && s < steps; ++s) warm_up(s);
    load_meta(0, ma);
    if (steps > 1) load_meta(1, mb);
    __syncthreads();
    decode(0, ma);
    __syncthreads();
    int s = 0;
    for (; s + 1 < steady_end; s += 2) {
      step(s, mb, ma, std::integral_constant<bool, true>{});
      step(s + 1, ma, mb, std::integral_constant<bool, true>{});
    }
    for (; s < steps; s += 2) {
      step(s, mb, ma, std::integral_constant<bool, false>{});
      if (s + 1 < steps) step(s + 1, ma, mb, std::integral_constant<bool, false>{});
    }
  }
}

// Y = fp16(sum over the splits of part[z]), the splits added in order
// (z = 0, 1, ...), so the result does not depend on timing. Four outputs
// per lane when the element count is a multiple of 4.
__global__ __launch_bounds__(256) void spmm_reduce_kernel(const float* __restrict__ part, int k_splits, long long count,
                                                          uint16_t* __restrict__ y) {
  const long long stride = (long long)gridDim.x * 256;
  if ((count & 3) == 0) {
    const long long n4 = count >> 2;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
      float4 s = reinterpret_cast<const float4*>(part)[i];
      for (int z = 1; z < k_splits; ++z) {
        const float4 p = reinterpret_cast<const float4*>(part + (size_t)z * (size_t)count)[i];
        s.x += p.x;
        s.y += p.y;
        s.z += p.z;
        s.w += p.w;
      }
      const uint32_t lo = __half_as_ushort(__float2half_rn(s.x)) | ((uint32_t)__half_as_ushort(__float2half_rn(s.y)) << 16);
      const uint32_t hi = __half_as_ushort(__float2half_rn(s.z)) | ((uint32_t)__half_as_ushort(__float2half_rn(s.w)) << 16);
      reinterpret_cast<uint2*>(y)[i] = make_uint2(lo, hi);
    }
  } else {
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < count; i += stride) {
      float s = part[i];
      for (int z = 1; z < k_splits; ++z) s += part[(size_t)z * (size_t)count + i];
      y[i] = __half_as_ushort(__float2half_rn(s));
    }
  }
}

int hip_fail(hipError_t e, const char* what) {
  return spdp::fail(SPDP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// The split-K partial sums of the prefill product: grown on demand, the
// old buffer kept until the handle is freed (a captured graph may still
// name it); no allocation while the stream is being captured.
int ensure_spmm_part(spdp_matrix* h, size_t bytes, hipStream_t stream) {
  if (bytes <= h->spmm_part_bytes) return SPDP_OK;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cs);
  if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
  if (cs != hipStreamCaptureStatusNone)
    return spdp::fail(SPDP_ERR_INVALID_ARG,
                      "the prefill split-K workspace is too small for this token count and the stream is "
                      "capturing; call spdp_spmm once with at least as many tokens before the capture");
  void* p = nullptr;
  e = hipMalloc(&p, bytes);
  if (e != hipSuccess)
    return e == hipErrorOutOfMemory ? spdp::fail(SPDP_ERR_OOM, "hipMalloc of the prefill workspace failed")
                                    : hip_fail(e, "hipMalloc");
  if (h->d_spmm_part) h->retired.push_back(h->d_spmm_part);
  h->d_spmm_part = p;
  h->spmm_part_bytes = bytes;
  return SPDP_OK;
}

}  // namespace

extern "C" int spdp_spmm(spdp_handle_t h, const uint16_t* X, int64_t n_tokens, uint16_t* Y, void* stream) {
  using spdp::fail;
  spdp::clear_error();
  if (!h) return fail(SPDP_ERR_INVALID_ARG, "handle is NULL");
  if (h->device < 0) return fail(SPDP_ERR_INVALID_ARG, "handle has no device copy");
  if (!X || !Y) return fail(SPDP_ERR_INVALID_ARG, "X or Y is NULL");
  if (n_tokens < 1) return fail(SPDP_ERR_INVALID_ARG, "n_tokens must be at least 1");
  if ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(Y)) & 15)
    return fail(SPDP_ERR_INVALID_ARG, "X and Y must be 16-byte aligned");
  {
    const uintptr_t x0 = reinterpret_cast<uintptr_t>(X), x1 = x0 + (uintptr_t)n_tokens * h->cols * 2;
    const uintptr_t y0 = reinterpret_cast<uintptr_t>(Y), y1 = y0 + (uintptr_t)n_tokens * h->rows * 2;
    if (x0 < y1 && y0 < x1) return fail(SPDP_ERR_INVALID_ARG, "X and Y overlap");
  }
  if (h->value_bits < 16) return fail(SPDP_ERR_UNSUPPORTED, "the prefill product takes fp16 Values, not codes");
  if (h->tile_m != kTM || h->tile_k < kKStep)
    return fail(SPDP_ERR_UNSUPPORTED, "the prefill product needs tile_m = 256 and tile_k >= 16");
  if ((n_tokens + kBN - 1) / kBN > 65535 || h->n_stripes > 0x7FFFFFFF)
    return fail(SPDP_ERR_UNSUPPORTED, "more than 65535 x 128 tokens");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != h->device) return fail(SPDP_ERR_INVALID_ARG, "current device differs from the handle's");
  SpmmArgs a;
  std::memset(&a, 0, sizeof(a));
  a.tile_offset = static_cast<const uint32_t*>(h->d_tile_offset);
  a.col_info = static_cast<const uint32_t*>(h->d_col_info);
  a.bitmap = static_cast<const uint64_t*>(h->d_bitmap);
  a.values = static_cast<const uint16_t*>(h->d_values);
  a.x = X;
  a.y = Y;
  a.n_tokens = n_tokens;
  a.rows = (int)h->rows;
  a.cols = (int)h->cols;
  a.tk_log2 = __builtin_ctz((unsigned)h->tile_k);
  a.n_colblocks = (int)h->n_colblocks;
  a.steps = (int)(h->n_colblocks * h->tile_k / kKStep);
  a.x_vec = h->cols % 8 == 0;
  a.y_vec = h->rows % 4 == 0;
  const long long tok_tiles = (n_tokens + kBN - 1) / kBN;
  auto st = static_cast<hipStream_t>(stream);
  // SPDP_SPMM_FORM (a testing aid): 1 the plain form, 2 the 128-token
  // warp-specialized form, 3 the 256-token one
  int form = 0;
  if (const char* env = std::getenv("SPDP_SPMM_FORM")) form = std::atoi(env);
  if (h->tile_k == kKStep && a.x_vec && form != 1) {
    // 256-token workgroups above 128 tokens when their grid, split, covers
    // at least half the CUs (the expansion of a GTile is paid once per
    // workgroup; below that the 128-token form's larger grid wins); split K
    // when the (stripe, token tile) grid leaves CUs idle, so that a split's
    // TileOffsets fit the LDS table, and with at least 8 GTiles per split
    // (40 for the 256-token form). A workgroup of either form holds its CU,
    // so the split never asks for more workgroups than there are CUs: a
    // second round for a few of them doubles the time. Measured (us; the
    // previous rule, 256-token workgroups only when two of them per CU were
    // left unsplit and the split rounded up -> this one): 11008x4096 at 128
    // / 256 / 512 tokens 66 / 108 / 148 -> 42 / 57 / 95, 8192x8192 at 512
    // 149 -> 105, 28672x8192 at 128 / 512 199 / 334 -> 145 / 294, 4096x4096
    // at 1024 90 -> 77.
    const int ncb = (int)h->n_colblocks;
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    const long long tiles256 = (n_tokens + kBN256 - 1) / kBN256;
    const long long wgs256 = h->n_stripes * tiles256;
    long long k256 = wgs256 < cus ? std::max<long long>(1, std::min<long long>(8, cus / wgs256)) : 1;
    k256 = std::min<long long>(k256, std::max(1, ncb / 40));
    const bool wide = form == 3 || (form != 2 && n_tokens > kBN && 2 * wgs256 * k256 >= cus);
    const long long tiles = wide ? tiles256 : tok_tiles;
    const long long wgs = h->n_stripes * tiles;
    long long k = wide ? k256 : wgs < cus ? std::max<long long>(1, std::min<long long>(8, cus / wgs)) : 1;
    if (!wide) k = std::min<long long>(k, std::max(1, ncb / 8));
    if (const char* env = std::getenv("SPDP_SPMM_SPLITS")) k = std::max(1, std::atoi(env));
    k = std::max<long long>(k, (ncb + kToCap - 2) / (kToCap - 1));
    k = std::min<long long>(k, ncb);
    const int sps = (int)((ncb + k - 1) / k);
    k = (ncb + sps - 1) / sps;  // every split non-empty
    if (k > 65535) return fail(SPDP_ERR_UNSUPPORTED, "the width needs more than 65535 splits");
    WsArgs wa;
    wa.s = a;
    wa.k_splits = (int)k;
    wa.sps = sps;
    wa.part = nullptr;
    if (k > 1) {
      const size_t bytes = (size_t)k * (size_t)n_tokens * (size_t)h->rows * sizeof(float);
      const int st_ok = ensure_spmm_part(h, bytes, st);
      if (st_ok != SPDP_OK) return st_ok;
      wa.part = static_cast<float*>(h->d_spmm_part);
    }
    const dim3 grid((unsigned)h->n_stripes, (unsigned)tiles, (unsigned)k);
    if (wide)
      hipLaunchKernelGGL(spmm_ws256_kernel, grid, dim3(kW256Waves * 64), 0, st, wa);
    else
      hipLaunchKernelGGL(spmm_ws_kernel, grid, dim3(kWsWaves * 64), 0, st, wa);
    if (k > 1) {
      e = hipGetLastError();
      if (e != hipSuccess) return hip_fail(e, "kernel launch");
      const long long count = n_tokens * h->rows;
      const long long per = (count & 3) == 0 ? count / 4 : count;
      const unsigned blocks = (unsigned)std::min<long long>(8192, (per + 255) / 256);
      hipLaunchKernelGGL(spmm_reduce_kernel, dim3(blocks), dim3(256), 0, st, wa.part, (int)k, count, Y);
    }
  } else {
    hipLaunchKernelGGL(spmm_kernel, dim3((unsigned)h->n_stripes, (unsigned)tok_tiles), dim3(kWaves * 64), 0, st, a);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return SPDP_OK;
}
