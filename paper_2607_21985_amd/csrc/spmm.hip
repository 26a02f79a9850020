// Prefill product on the Tiled-CBC arrays (Sec. 4.3): Y = X W_sp^T for N
// tokens with static pruning only (no activation test), on gfx950's matrix
// cores. The weights stay in the decode format -- the same handle serves
// both phases -- and are expanded tile by tile into a dense operand in LDS
// (the paper's layout-alignment stage), then multiplied with
// v_mfma_f32_32x32x16_f16 (fp16 operands, fp32 accumulation).
//
// Workgroup (4 waves) = one 256-row stripe x 128 tokens. Per k-step of 16
// columns (one GTile of a 256 x 16 tiling):
//   1. decode: wave w expands columns 4w .. 4w+3 of the step, all four
//      64-row bitmap words each: lane i of word v takes row 64v + i, its
//      value at the word's masked popcount below bit i plus the popcounts of
//      the column's earlier words (HAD-SMBD, Sec. 4.2.1), or 0 where the bit
//      is clear; the four columns of a row go to LDS as one 8-byte store
//      (row-major dense tile, 16 fp16 per row, rows padded to 40 bytes);
//   2. multiply: wave w owns tokens 32w .. 32w+31; its B operand (16 k x
//      32 tokens) is read straight from X (lane l: token l mod 32, eight
//      consecutive k), and for each of the eight 32-row blocks of the
//      stripe one MFMA adds A (32 rows x 16 k, two 8-byte LDS reads per
//      lane) times B into that block's 32 x 32 accumulators.
// The dense tile is double-buffered, so one barrier per k-step separates a
// step's LDS writes from the other waves' reads. Every k-step's metadata,
// values and X block are requested one step ahead, while the current
// step's MFMAs run.

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstring>

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

// What one wave fetches for one k-step: its four columns' values (one per
// lane and bitmap word, 0 where the bit is clear) and its B operand.
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
// The pipelined form for 256 x 16 GTiles and a width that is a multiple of
// 8 (every Llama shape): each k-step is one GTile, and everything a step
// reads from memory -- the GTile's padded values (one contiguous run), its
// 16 columns' bitmap words and ColInfo, and the 128 x 16 block of X -- is
// copied into a ring of kRing LDS slots by global->LDS DMA, kRing steps
// ahead, so that no wave waits on memory for the decode. Per wave and step:
// two 16-byte DMA loads of values (the GTile's values in 16-byte chunks over
// 4 waves x 2 loads x 64 lanes; lanes past the end re-read the last chunk),
// one 4-byte DMA load of bitmap words or ColInfo, one 16-byte DMA load of
// its own 32 tokens of X: four loads, so "step s has landed" is "at most
// 4 x (later steps requested) loads outstanding". Step s: the MFMAs of step
// s (dense tile s & 1, B operand from the wave's own X rows of slot s), then
// the DMA of step s + kRing into slot s (its values, bitmaps and ColInfo
// were decoded in step s - 1, its X rows were just read), then the decode of
// step s + 1 into dense tile (s + 1) & 1 while the MFMAs run, then one
// barrier.

constexpr int kRing = 4;
constexpr int kMetaBytes = 1024;               // bitmaps (512 B), ColInfo (64 B), DMA spill
constexpr int kValBytes = kTM * kKStep * 2;    // a dense GTile's worth of values
constexpr int kXBytes = kBN * kKStep * 2;      // 128 tokens x 16 columns
constexpr int kSlotBytes = kMetaBytes + kValBytes + kXBytes;

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
constexpr int kDmaPerStep = 4;

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void spmm_ring_kernel(SpmmArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char ring[kRing][kSlotBytes];
  __shared__ __attribute__((aligned(16))) unsigned char tile[2][kTileBytes];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = blockIdx.x;
  const long long nb0 = (long long)blockIdx.y * kBN;
  const int khalf = (lane >> 5) * 8;
  const int steps = a.steps;
  const const_ptr<uint32_t> to_s = (const_ptr<uint32_t>)a.tile_offset;
  const uint32_t g0 = (uint32_t)r * (uint32_t)a.n_colblocks;
  // this workgroup's 128 tokens of X (tokens past the end re-read the last)
  const uint16_t* const xblk = a.x + nb0 * (long long)a.cols;
  const long long left = a.n_tokens - nb0;
  // X DMA: lane l of wave w brings token 32w + l / 2, columns 8 (l & 1) ..
  // + 8 of the step, to byte 1024 w + 16 l of the slot's X block
  const int xt = 32 * wave + (lane >> 1);
  const uint32_t x_row = (uint32_t)((xt < left ? xt : left - 1) * (long long)a.cols * 2);

  auto issue = [&](int s) __attribute__((always_inline)) {
    unsigned char* slot = ring[s % kRing];
    const uint32_t g = g0 + (uint32_t)s;
    const uint32_t t0 = to_s[g], t1 = to_s[g + 1];
    const uint32_t last = t1 > t0 ? (t1 - t0) / 8u - 1u : 0u;  // last 16-byte chunk of the values
    const uint32_t vbase = lds_addr(slot + kMetaBytes);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t q = (uint32_t)((i * kWaves + wave) * 64 + lane);
      dma16(a.values, 2u * t0 + 16u * (q < last ? q : last),
            (uint32_t)__builtin_amdgcn_readfirstlane((int)(vbase + (uint32_t)(i * kWaves + wave) * 1024u)));
    }
    // waves 0, 1: the 16 columns' bitmap words (512 bytes); wave 2 the
    // ColInfo (64 bytes; its other lanes re-read it); wave 3 re-reads it too
    const uint32_t mbase = lds_addr(slot) + 256u * (uint32_t)wave;
    if (wave < 2)
      dma4(a.bitmap, g * 512u + 256u * (uint32_t)wave + 4u * (uint32_t)lane,
           (uint32_t)__builtin_amdgcn_readfirstlane((int)mbase));
    else
      dma4(a.col_info, g * 64u + 4u * (uint32_t)(lane & 15), (uint32_t)__builtin_amdgcn_readfirstlane((int)mbase));
    const uint32_t xk = (uint32_t)(s * kKStep + 8 * (lane & 1));
    // columns past the width: any valid 16 bytes (the weights there are 0;
    // the B operand is cleared after the read)
    const uint32_t xoff = x_row + 2u * (xk < (uint32_t)a.cols ? xk : 0u);
    dma16(xblk, xoff, (uint32_t)__builtin_amdgcn_readfirstlane((int)lds_addr(slot + kMetaBytes + kValBytes + 1024 * wave)));
  };
  // "step s landed": at most kDmaPerStep x (steps requested after s) loads
  // in flight, the count being min(kRing - 1, steps - 1 - s) in the steady state
  auto wait_landed = [&](int later) __attribute__((always_inline)) {
    if (later >= 3)
      wait_vmcnt<3 * kDmaPerStep>();
    else if (later == 2)
      wait_vmcnt<2 * kDmaPerStep>();
    else if (later == 1)
      wait_vmcnt<kDmaPerStep>();
    else
      wait_vmcnt<0>();
  };
  static_assert(kRing == 4, "wait_landed counts up to three later steps");
  // decode of step s (slot s % kRing) into dense tile `t`: wave w expands
  // columns 4w .. 4w + 3, lane i of word v giving row 64 v + i. ColInfo and
  // the bitmap words come from scalar loads (the step's DMA has brought
  // their lines into L2) straight into scalar registers, where they serve as
  // mbcnt masks and as the select mask of the lanes' values; the values come
  // from the slot.
  const const_ptr<uint32_t> ci_s = (const_ptr<uint32_t>)a.col_info;
  const const_ptr<uint64_t> bm_s = (const_ptr<uint64_t>)a.bitmap;
  struct Meta {
    uint32_t ci[4];
    uint64_t words[4][4];
  };
  // requested one step ahead of its decode, so that the scalar loads' round
  // trip overlaps the previous step's work
  auto meta_of = [&](int s, Meta& m) __attribute__((always_inline)) {
    const uint32_t col0 = (g0 + (uint32_t)s) * (uint32_t)kKStep + 4u * (uint32_t)wave;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      m.ci[jj] = ci_s[col0 + jj];
#pragma unroll
      for (int v = 0; v < 4; ++v) m.words[jj][v] = bm_s[(size_t)(col0 + jj) * 4 + v];
    }
  };
  auto decode = [&](int s, const Meta& m, unsigned char* t) __attribute__((always_inline)) {
    const unsigned char* slot = ring[s % kRing];
    const uint32_t (&ci)[4] = m.ci;
    const uint64_t (&words)[4][4] = m.words;
    const uint32_t vb = lds_addr(slot + kMetaBytes);
    uint32_t h[4][4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      uint32_t base = vb + 2u * (ci[jj] >> 16);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const uint64_t word = words[jj][v];
        const uint32_t hv =
            *(const __attribute__((address_space(3))) uint16_t*)(uintptr_t)(base + 2u * mbcnt64(word));
        // the lane's value where its bit is set, else 0 (the word as the select mask)
        uint32_t sel;
        asm("v_cndmask_b32_e64 %0, 0, %1, %2" : "=v"(sel) : "v"(hv), "s"(word));
        h[v][jj] = sel;
        base += 2u * (uint32_t)__builtin_popcountll(word);
      }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v)
      *reinterpret_cast<uint2*>(t + (64 * v + lane) * kRowBytes + 8 * wave) =
          make_uint2(h[v][0] | (h[v][1] << 16), h[v][2] | (h[v][3] << 16));
  };

  float16v acc[kBlocks];
#pragma unroll
  for (int i = 0; i < kBlocks; ++i) acc[i] = float16v{};

  // prologue: the first kRing steps requested, step 0 decoded, step 1 landed
  for (int s = 0; s < kRing && s < steps; ++s) issue(s);
  Meta meta;
  meta_of(0, meta);
  wait_landed(min(kRing - 1, steps - 1));
  __syncthreads();
  decode(0, meta, tile[0]);
  if (steps > 1) meta_of(1, meta);
  wait_landed(min(kRing - 2, steps - 2));
  __syncthreads();

  for (int s = 0; s < steps; ++s) {
    unsigned char* slot = ring[s % kRing];
    const unsigned char* t = tile[s & 1];
    // B operand: this wave's 32 tokens, 8 columns, from its own X rows
    half8 b = *reinterpret_cast<const half8*>(slot + kMetaBytes + kValBytes +
                                              (32 * wave + (lane & 31)) * 32 + 2 * khalf);
    if (s * kKStep + khalf >= a.cols) b = half8{0, 0, 0, 0, 0, 0, 0, 0};
    half8 av[kBlocks];
#pragma unroll
    for (int i = 0; i < kBlocks; ++i) {
      const unsigned char* p = t + (32 * i + (lane & 31)) * kRowBytes + 2 * khalf;
      const uint2 lo = *reinterpret_cast<const uint2*>(p);
      const uint2 hi = *reinterpret_cast<const uint2*>(p + 8);
      av[i] = __builtin_bit_cast(half8, make_uint4(lo.x, lo.y, hi.x, hi.y));
    }
#pragma unroll
    for (int i = 0; i < kBlocks; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[i], b, acc[i], 0, 0, 0);
    // the slot's X rows have been read (the operands are in registers); its
    // values and metadata were decoded before the last barrier
    if (s + kRing < steps) issue(s + kRing);
    if (s + 1 < steps) decode(s + 1, meta, tile[(s + 1) & 1]);
    // step s + 2 (decoded in the next iteration) has landed: the steps
    // requested after it are s + 3 .. min(s + kRing, steps - 1)
    if (s + 2 < steps) {
      wait_landed(min(kRing - 2, steps - 1 - (s + 2)));
      meta_of(s + 2, meta);
    }
    __syncthreads();
  }

  const long long n = nb0 + 32 * wave + (lane & 31);
  if (n >= a.n_tokens) return;
  uint16_t* const yrow = a.y + n * (long long)a.rows;
#pragma unroll
  for (int i = 0; i < kBlocks; ++i) {
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const int m = r * kTM + 32 * i + 8 * grp + 4 * (lane >> 5);
      uint16_t hh[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) hh[e] = __half_as_ushort(__float2half_rn(acc[i][4 * grp + e]));
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

int hip_fail(hipError_t e, const char* what) {
  return spdp::fail(SPDP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
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
  const dim3 grid((unsigned)h->n_stripes, (unsigned)((n_tokens + kBN - 1) / kBN));
  // the pipelined form for 256 x 16 GTiles and 16-byte X rows; the plain one otherwise
  if (h->tile_k == kKStep && a.x_vec)
    hipLaunchKernelGGL(spmm_ring_kernel, grid, dim3(kWaves * 64), 0, static_cast<hipStream_t>(stream), a);
  else
    hipLaunchKernelGGL(spmm_kernel, grid, dim3(kWaves * 64), 0, static_cast<hipStream_t>(stream), a);
  e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return SPDP_OK;
}
