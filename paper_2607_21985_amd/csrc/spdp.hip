// Device side of libspdp for gfx950 (MI355X): the fused decode-time spMspV
// kernel over Tiled-CBC weights (Sec. 4.2) and the C-ABI entry points that
// own device memory.
//
// One launch per call does the whole path:
//   1. activity: each wave reads its K range of the activations and takes
//      the strict magnitude test |x| > t as an integer compare on fp16 bits;
//      64-lane ballots (union over the batch) compact the active columns into
//      a per-wave list in LDS (Sec. 4.2, XTile loading and the
//      activation-aware selection of GTile loading);
//   2. metadata then data (Sec. 4.2.2): ColInfo and TileOffset of the range
//      arrive in the same round trip as the activations; the list then
//      drives batches of 8 active columns whose padded values (16-byte vector
//      loads, two columns per load instruction) and bitmap words stream into
//      registers three batches ahead of the decode; a batch moves to LDS
//      right before it is decoded;
//   3. bitmap decode (HAD-SMBD, Sec. 4.2.1): lane i owns row 64w+i of bitmap
//      word w; its value sits at the masked popcount of the word below bit i
//      (v_mbcnt_lo/hi, the MaskedPopcount of the paper) plus the popcount of
//      the earlier words, and the word itself (read out of the batch's
//      registers with v_readlane) is the execution mask, so rows without a
//      nonzero issue no LDS read and no FMA;
//   4. accumulate in fp32 on the vector ALUs with fp16 operands (v_fma_mix),
//      no matrix cores (Sec. 3.3 challenge 2, Sec. 4.2 step 5);
//   5. split-K (Sec. 4.2.3): the workgroups of a row stripe cover disjoint K
//      segments; each reduces its 4 waves in LDS. Every segment but the last
//      stores its fp32 partial sums to a workspace, each value paired with
//      the stripe's phase number in one 8-byte store; the last segment's
//      workgroup loads the other segments' partials until every one carries
//      the current phase, adds them in segment order (its own last), writes
//      fp16 Y (round to nearest even) and advances the stripe's phase for
//      the next call. No counter, no fence, no host-side state: a partial
//      is usable as soon as its own store has landed, and a captured graph
//      replays correctly.

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <new>

#include "internal.h"

namespace {

constexpr int kWaves = 4;                 // waves per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxWords = 4;              // tile_m <= 256: at most 4 bitmap words per column
constexpr int kSlotBytes = 64 * kMaxWords * 2;  // LDS slot: one column of one stripe (fp16)
constexpr int kBatch = 8;                 // active columns per pipeline stage of a wave
constexpr int kQuad = 4;                  // columns decoded together
constexpr int kMaxWaveCols = 128;         // columns of one wave's K range
constexpr int kDepth = 2;                 // batches whose values are in flight per wave
constexpr int kMaxBatch = 32;
constexpr int kDummyBatch = kMaxWaveCols / kBatch;  // LDS batch of all-zero entries

struct KernelArgs {
  const uint32_t* tile_offset;
  const uint32_t* col_info;
  const uint64_t* bitmap;
  const uint16_t* values;
  const uint16_t* x;
  uint16_t* y;
  // [segments][batch][n_stripes * tile_m]: {fp32 bits, phase} pairs
  unsigned long long* partials;
  uint32_t* phase;     // [n_stripes], never 0 (the workspace starts zeroed)
  int rows, cols;
  int tile_m, tk_log2, n_colblocks, n_stripes;
  int batch;
  int code;       // threshold code: active iff code < (x & 0x7fff) <= 0x7c00
  int wave_cols;  // columns per wave (multiple of 16, <= kMaxWaveCols)
  int segments;   // workgroups per row stripe
  uint32_t zero_col;  // column index whose bitmap lies in the zeroed tail padding
};

// LDS use: one value slot buffer per wave (the batch being decoded; the
// batches in flight live in registers).
constexpr int kValBufBytes = kWaves * kBatch * kSlotBytes;

template <int NB>
struct Smem {
  static constexpr int kSlice = NB < 4 ? NB : 4;  // tokens per cross-wave reduction pass
  static constexpr int kRed = kWaves * kSlice * 256 * 4;
  static_assert(kRed <= kValBufBytes, "reduction reuses the value buffer");
};

__device__ __forceinline__ uint32_t mbcnt64(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return __half2float(__ushort_as_half((unsigned short)h));
}

// Pointers into the constant address space: reads through them are scalar
// loads.
template <class T>
using const_ptr = const __attribute__((address_space(4))) T*;

// One column of one token: acc[w] += f32(v[w]) * f32(x) in the lanes whose
// bit is set in word w, where v[w] is fp16 bits and x the low (XHI false) or
// high (XHI true) fp16 half of xpair. The whole column is one block so that
// nothing else runs under the narrowed EXEC: save EXEC while ANDing it with
// the first word, AND the saved mask with each later word, restore at the end
// (one scalar instruction per word, no branch).
#define SPDP_FMA(W, SEL) "v_fma_mix_f32 %[a" #W "], %[v" #W "], %[x], %[a" #W "] " SEL "\n\t"
#define SPDP_COLUMN(SEL)                                                                              \
  if constexpr (WPC == 1) {                                                                           \
    asm volatile("s_and_saveexec_b64 %[sv], %[m0]\n\t" SPDP_FMA(0, SEL) "s_mov_b64 exec, %[sv]"      \
                 : [a0] "+v"(acc[0][0]), [sv] "=&s"(save)                                             \
                 : [m0] "s"(m[0]), [v0] "v"(v[0]), [x] "v"(xpair)                                     \
                 : "scc");                                                                            \
  } else if constexpr (WPC == 2) {                                                                    \
    asm volatile("s_and_saveexec_b64 %[sv], %[m0]\n\t" SPDP_FMA(0, SEL)                              \
                 "s_and_b64 exec, %[sv], %[m1]\n\t" SPDP_FMA(1, SEL) "s_mov_b64 exec, %[sv]"          \
                 : [a0] "+v"(acc[0][0]), [a1] "+v"(acc[1][0]), [sv] "=&s"(save)                       \
                 : [m0] "s"(m[0]), [m1] "s"(m[1]), [v0] "v"(v[0]), [v1] "v"(v[1]), [x] "v"(xpair)     \
                 : "scc");                                                                            \
  } else if constexpr (WPC == 3) {                                                                    \
    asm volatile("s_and_saveexec_b64 %[sv], %[m0]\n\t" SPDP_FMA(0, SEL)                              \
                 "s_and_b64 exec, %[sv], %[m1]\n\t" SPDP_FMA(1, SEL)                                  \
                 "s_and_b64 exec, %[sv], %[m2]\n\t" SPDP_FMA(2, SEL) "s_mov_b64 exec, %[sv]"          \
                 : [a0] "+v"(acc[0][0]), [a1] "+v"(acc[1][0]), [a2] "+v"(acc[2][0]), [sv] "=&s"(save) \
                 : [m0] "s"(m[0]), [m1] "s"(m[1]), [m2] "s"(m[2]), [v0] "v"(v[0]), [v1] "v"(v[1]),    \
                   [v2] "v"(v[2]), [x] "v"(xpair)                                                     \
                 : "scc");                                                                            \
  } else {                                                                                            \
    static_assert(WPC == 4, "at most four bitmap words per column");                                  \
    asm volatile("s_and_saveexec_b64 %[sv], %[m0]\n\t" SPDP_FMA(0, SEL)                              \
                 "s_and_b64 exec, %[sv], %[m1]\n\t" SPDP_FMA(1, SEL)                                  \
                 "s_and_b64 exec, %[sv], %[m2]\n\t" SPDP_FMA(2, SEL)                                  \
                 "s_and_b64 exec, %[sv], %[m3]\n\t" SPDP_FMA(3, SEL) "s_mov_b64 exec, %[sv]"          \
                 : [a0] "+v"(acc[0][0]), [a1] "+v"(acc[1][0]), [a2] "+v"(acc[2][0]),                  \
                   [a3] "+v"(acc[3][0]), [sv] "=&s"(save)                                             \
                 : [m0] "s"(m[0]), [m1] "s"(m[1]), [m2] "s"(m[2]), [m3] "s"(m[3]), [v0] "v"(v[0]),    \
                   [v1] "v"(v[1]), [v2] "v"(v[2]), [v3] "v"(v[3]), [x] "v"(xpair)                     \
                 : "scc");                                                                            \
  }
template <int WPC, bool XHI>
__device__ __forceinline__ void masked_fma_column(float (&acc)[WPC][1], const uint32_t (&v)[WPC],
                                                  uint32_t xpair, const uint64_t (&m)[WPC]) {
  uint64_t save;
  if constexpr (XHI) {
    SPDP_COLUMN("op_sel:[0,1,0] op_sel_hi:[1,1,0]")
  } else {
    SPDP_COLUMN("op_sel_hi:[1,1,0]")
  }
}
#undef SPDP_COLUMN
#undef SPDP_FMA

// The kernel's argument block, read again from the kernel-argument segment
// through a pointer the compiler cannot see through: fields used only after
// the main loop are loaded there instead of holding scalar registers
// throughout it.
template <class Args>
__device__ __forceinline__ const_ptr<Args> reload_args() {
  auto p = (const_ptr<Args>)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(p));
  return p;
}

// NB: tokens per call rounded up to a power of two; WPC: bitmap words per
// column (tile_m / 64).
template <int NB, int WPC>
__global__ __launch_bounds__(kThreads) void spmspv_kernel(KernelArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char valbuf[kValBufBytes];
  // one entry per active column, in activity order: {byte offset of the
  // column's values, column index into ColInfo/bitmap << 6 | index of its
  // last 16-byte chunk}; batch kDummyBatch holds entries that load nothing
  // of use (see below)
  __shared__ uint2 ent_s[kWaves][kMaxWaveCols + kBatch];
  __shared__ __attribute__((aligned(16))) uint16_t xs_s[kWaves][kMaxWaveCols * NB];
  __shared__ int s_last;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int seg = blockIdx.x;
  const int r = blockIdx.y;
  const int tk_mask = (1 << a.tk_log2) - 1;
  const int g_row = r * a.n_colblocks;

  uint2* ent_l = ent_s[wave];
  uint16_t* xs_l = xs_s[wave];
  unsigned char* my_val = valbuf + wave * (kBatch * kSlotBytes);

  float acc[WPC][NB];
#pragma unroll
  for (int w = 0; w < WPC; ++w)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[w][b] = 0.0f;

  // the stripe's phase: written by the previous call's last segment, read
  // by every workgroup of the stripe before any of them publishes
  const uint32_t phase = ((const_ptr<uint32_t>)a.phase)[r];
  const int k_begin = (seg * kWaves + wave) * a.wave_cols;
  const int range = max(0, min(a.wave_cols, a.cols - k_begin));

  // ---- 1. the wave's K range: activations and column metadata in one round
  // trip (ColInfo/TileOffset are fetched for every column of the range, which
  // removes a dependent memory round trip; their cache lines are shared by
  // neighbouring columns, so little extra traffic results).
  constexpr int kChunks = kMaxWaveCols / 64;
  uint32_t ci[kChunks], to[kChunks], colx[kChunks], xb[kChunks][NB];
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int off = 64 * c + lane;
    const bool in = off < range;
    const int k = k_begin + (in ? off : 0);
    const int g = g_row + (k >> a.tk_log2);
    colx[c] = ((uint32_t)g << a.tk_log2) + (uint32_t)(k & tk_mask);
    ci[c] = 0u;
    to[c] = 0u;
    if (64 * c < range) {
      ci[c] = a.col_info[colx[c]];
      to[c] = a.tile_offset[g];
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) xb[c][b] = (in && b < a.batch) ? a.x[(size_t)b * a.cols + k] : 0u;
  }
  int n_act = 0;
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int off = 64 * c + lane;
    const bool in = off < range;
    uint64_t act = 0;
    bool on[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int mag = (int)(xb[c][b] & 0x7FFFu);
      on[b] = in && b < a.batch && mag > a.code && mag <= 0x7C00;
      act |= __builtin_amdgcn_ballot_w64(on[b]);
    }
    if ((act >> lane) & 1) {
      const int pos = n_act + (int)mbcnt64(act);
      const uint32_t chunks = ((ci[c] & 0xFFFFu) + 7u) >> 3;
      ent_l[pos] = make_uint2(2u * (to[c] + (ci[c] >> 16)), (colx[c] << 6) | (chunks ? chunks - 1u : 0u));
#pragma unroll
      for (int b = 0; b < NB; ++b) xs_l[pos * NB + b] = on[b] ? (uint16_t)xb[c][b] : (uint16_t)0;
    }
    n_act += __builtin_popcountll(act);
  }
  // Pad the last batch with entries that read an all-zero bitmap (in the
  // bitmap array's zeroed tail) and no values: they decode to nothing.
  // The dummy batch is all such entries; stages past the last batch load it.
  if (lane < ((kBatch - (n_act & (kBatch - 1))) & (kBatch - 1))) {
    ent_l[n_act + lane] = make_uint2(0u, a.zero_col << 6);
  }
  if (lane < kBatch) {
    ent_l[kDummyBatch * kBatch + lane] = make_uint2(0u, a.zero_col << 6);
  }

  // ---- 2. pipeline over batches of kBatch active columns: while batch i is
  // decoded, batch i+1's values and bitmaps are already streaming into LDS.
  const int n_batches = (n_act + kBatch - 1) / kBatch;
  const int hsel = lane >> 5;
  const int q = lane & 31;
  const unsigned char* value_bytes = reinterpret_cast<const unsigned char*>(a.values);
  const unsigned char* bitmap_bytes = reinterpret_cast<const unsigned char*>(a.bitmap);

  // A stage holds one batch in registers. Values: lane l of load pr has 16
  // bytes of column 2pr + (l >= 32), chunk l & 31; lanes past a column's end
  // re-read its last chunk (a line the column loads anyway) and what they
  // leave in the slot is never read. Bitmaps: lane l holds dword l % (2 WPC)
  // of column (l / (2 WPC)) % 8, so the decode reads the batch's words out of
  // that register. A stage past the last batch loads the dummy batch (all
  // lanes read the same 16 bytes of values and an all-zero bitmap), so every
  // stage issues the same loads and the in-order wait counts release exactly
  // the oldest stage. Offsets are 32-bit from a wave-uniform base (the value
  // and bitmap arrays stay below 4 GiB).
  static_assert(kBatch == 8, "a stage is four 16-byte loads per lane");
  static_assert(kBatch * 2 * WPC <= 64, "a batch's bitmap words fit one dword per lane");
  const uint32_t bm_lane_off = (uint32_t)(lane % (2 * WPC)) * 4u;
  const int bm_col = (lane / (2 * WPC)) & (kBatch - 1);
#define SPDP_LOAD(E, V) \
  V = *reinterpret_cast<const uint4*>(value_bytes + ((E).x + (min((uint32_t)q, (E).y & 63u) << 4)))
#define SPDP_ISSUE(I, V)                                                                          \
  do {                                                                                            \
    const int bi_ = (I) < n_batches ? (I) : kDummyBatch;                                          \
    const uint2 e0_ = ent_l[bi_ * kBatch + 0 + hsel];                                             \
    const uint2 e1_ = ent_l[bi_ * kBatch + 2 + hsel];                                             \
    const uint2 e2_ = ent_l[bi_ * kBatch + 4 + hsel];                                             \
    const uint2 e3_ = ent_l[bi_ * kBatch + 6 + hsel];                                             \
    const uint32_t bcol_ = ent_l[bi_ * kBatch + bm_col].y >> 6;                                   \
    SPDP_LOAD(e0_, V##0);                                                                         \
    SPDP_LOAD(e1_, V##1);                                                                         \
    SPDP_LOAD(e2_, V##2);                                                                         \
    SPDP_LOAD(e3_, V##3);                                                                         \
    V##b = *reinterpret_cast<const uint32_t*>(bitmap_bytes + (bcol_ * (WPC * 8u) + bm_lane_off)); \
  } while (0)
#define SPDP_TO_LDS(V, BM)                                                                           \
  do {                                                                                            \
    *reinterpret_cast<uint4*>(my_val + 0 * kSlotBytes + 16 * lane) = V##0;                        \
    *reinterpret_cast<uint4*>(my_val + 2 * kSlotBytes + 16 * lane) = V##1;                        \
    *reinterpret_cast<uint4*>(my_val + 4 * kSlotBytes + 16 * lane) = V##2;                        \
    *reinterpret_cast<uint4*>(my_val + 6 * kSlotBytes + 16 * lane) = V##3;                        \
    BM = V##b;                                                                                    \
  } while (0)

  // Decode of batch i: its values are in the wave's LDS slots and its bitmap
  // words in bm (one dword per lane, see above): v_readlane moves them to
  // scalar registers, where they serve directly as MaskedPopcount masks and
  // EXEC masks.
  auto decode_quad = [&](int i, int u0, uint32_t bm) __attribute__((always_inline)) {
    uint64_t words[kQuad][WPC];
#pragma unroll
    for (int c = 0; c < kQuad; ++c)
#pragma unroll
      for (int w = 0; w < WPC; ++w) {
        const int l = (u0 + c) * 2 * WPC + 2 * w;
        words[c][w] = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)bm, l) |
                      ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)bm, l + 1) << 32);
      }
    // 3. bitmap decode: a row's value sits at the MaskedPopcount of its word
    // below the lane plus the popcounts of the column's earlier words
    uint32_t vb[kQuad][WPC];
#pragma unroll
    for (int c = 0; c < kQuad; ++c) {
      const uint16_t* slot = reinterpret_cast<const uint16_t*>(my_val + (u0 + c) * kSlotBytes);
      uint32_t prefix = 0;
#pragma unroll
      for (int w = 0; w < WPC; ++w) {
        vb[c][w] = slot[prefix + mbcnt64(words[c][w])];
        prefix += (uint32_t)__builtin_popcountll(words[c][w]);
      }
    }
    // 4. accumulate where the bitmap bit is set: for one token the words
    // become EXEC around single FMAs (no branch, no select); for more tokens
    // the compiler's FMA-plus-select on the word is used
    const int xrow = (i * kBatch + u0) * NB;
    // one token: the group's fp16 activations in one LDS read
    uint2 xq = make_uint2(0u, 0u);
    if constexpr (NB == 1) {
      if constexpr (kQuad == 4)
        xq = *reinterpret_cast<const uint2*>(&xs_l[xrow]);
      else
        xq.x = *reinterpret_cast<const uint32_t*>(&xs_l[xrow]);
    }
#pragma unroll
    for (int c = 0; c < kQuad; ++c) {
      if constexpr (NB == 1) {
        const uint32_t xpair = c < 2 ? xq.x : xq.y;
        if (c & 1)
          masked_fma_column<WPC, true>(acc, vb[c], xpair, words[c]);
        else
          masked_fma_column<WPC, false>(acc, vb[c], xpair, words[c]);
      } else {
        float xv[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) xv[b] = half_bits_to_float(xs_l[xrow + c * NB + b]);
#pragma unroll
        for (int w = 0; w < WPC; ++w)
          if (__builtin_amdgcn_inverse_ballot_w64(words[c][w])) {
            const float v = half_bits_to_float(vb[c][w]);
#pragma unroll
            for (int b = 0; b < NB; ++b) acc[w][b] = __builtin_fmaf(v, xv[b], acc[w][b]);
          }
      }
    }
  };
  // A batch is kBatch / kQuad groups; a group holding only padding entries
  // (all-zero words) is skipped.
  static_assert(kQuad == 2 || kQuad == 4, "columns are decoded in pairs or quads");
  auto decode = [&](int i, uint32_t bm) __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < kBatch / kQuad; ++g)
      if (g == 0 || n_act - i * kBatch > g * kQuad) decode_quad(i, g * kQuad, bm);
  };

  // kDepth batches in flight: a stage holds batch i while the next kDepth-1
  // batches stream; a batch moves to LDS right before its decode. The loop has
  // a single exit and every path through it issues the same loads, so the
  // waits at its head count exactly one stage. The stages must be issued in
  // order (the waits count loads in order), so the scheduler may not
  // interleave them.
  static_assert(kDepth == 2 || kDepth == 3, "the loop below is unrolled for two or three stages");
  if (n_batches > 0) {
    uint4 s00, s01, s02, s03, s10, s11, s12, s13;
    uint32_t s0b, s1b, bm;
    SPDP_ISSUE(0, s0);
    __builtin_amdgcn_sched_barrier(0);
    SPDP_ISSUE(1, s1);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (kDepth == 2) {
      for (int i = 0; i < n_batches; i += 2) {
        SPDP_TO_LDS(s0, bm);
        SPDP_ISSUE(i + 2, s0);
        __builtin_amdgcn_sched_barrier(0);
        decode(i, bm);
        SPDP_TO_LDS(s1, bm);
        SPDP_ISSUE(i + 3, s1);
        __builtin_amdgcn_sched_barrier(0);
        if (i + 1 < n_batches) decode(i + 1, bm);
      }
    } else {
      uint4 s20, s21, s22, s23;
      uint32_t s2b;
      SPDP_ISSUE(2, s2);
      __builtin_amdgcn_sched_barrier(0);
      for (int i = 0; i < n_batches; i += 3) {
        SPDP_TO_LDS(s0, bm);
        SPDP_ISSUE(i + 3, s0);
        __builtin_amdgcn_sched_barrier(0);
        decode(i, bm);
        SPDP_TO_LDS(s1, bm);
        SPDP_ISSUE(i + 4, s1);
        __builtin_amdgcn_sched_barrier(0);
        if (i + 1 < n_batches) decode(i + 1, bm);
        SPDP_TO_LDS(s2, bm);
        SPDP_ISSUE(i + 5, s2);
        __builtin_amdgcn_sched_barrier(0);
        if (i + 2 < n_batches) decode(i + 2, bm);
      }
    }
  }
#undef SPDP_LOAD
#undef SPDP_ISSUE
#undef SPDP_TO_LDS

  // ---- 5. reduce the 4 waves in LDS and publish this segment's partial
  // sums: device-coherent 8-byte stores, so that value and tag land together
  // and can be read from another XCD
  const_ptr<KernelArgs> ka = reload_args<KernelArgs>();
  const int mpad = ka->n_stripes * ka->tile_m;
  const int n_seg = ka->segments;
  const int nb = ka->batch;
  const int row = threadIdx.x;
  float* red = reinterpret_cast<float*>(valbuf);
  constexpr int kSlice = Smem<NB>::kSlice;
  unsigned long long* dst = ka->partials + (size_t)seg * nb * mpad + (size_t)r * ka->tile_m + row;
  const unsigned long long tag = (unsigned long long)phase << 32;
#pragma unroll
  for (int b0 = 0; b0 < NB; b0 += kSlice) {
    __syncthreads();
#pragma unroll
    for (int w = 0; w < WPC; ++w)
#pragma unroll
      for (int bb = 0; bb < kSlice; ++bb) red[(wave * kSlice + bb) * 256 + 64 * w + lane] = acc[w][b0 + bb];
    __syncthreads();
#pragma unroll
    for (int bb = 0; bb < kSlice; ++bb) {
      if (row < 64 * WPC && b0 + bb < nb) {
        float s = 0.0f;
#pragma unroll
        for (int wv = 0; wv < kWaves; ++wv) s += red[(wv * kSlice + bb) * 256 + row];
        __hip_atomic_store(dst + (size_t)(b0 + bb) * mpad, tag | __float_as_uint(s), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }

  // ---- the stripe's last n_red segments gather: reducer j owns the 64-row
  // blocks w = j, j + n_red, ...; its four waves split the segments (wave g
  // takes segments g, g+4, ...), request all of a chunk of them at once,
  // request again those not yet tagged with this call's phase, and add them
  // in order; the four wave sums are added in wave order, so the result does
  // not depend on timing. The workgroups of lower segments of the stripe were
  // dispatched before these, so the wait ends; a bound on the rounds still
  // makes every wave exit (the rows then read NaN).
  const int n_red = min(n_seg, WPC);
  const int jr = seg - (n_seg - n_red);
  if (jr < 0) return;
  // A round requests kJ of the wave's segments for every token at once
  // (about kGather partials in flight per lane).
  constexpr int kGather = 12;
  constexpr int kJ = NB >= kGather ? 1 : kGather / NB;
  constexpr int kMaxRounds = 1 << 22;
  const int rows = ka->rows;
  for (int w = jr; w < WPC; w += n_red) {
    const int m = r * ka->tile_m + 64 * w + lane;
    const bool live = m < rows;
    const unsigned long long* src = ka->partials + (live ? m : 0);
    float sums[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) sums[b] = 0.0f;
    if (live) {
      bool lost = false;
      auto part = [&](int sg, int b) {
        return __hip_atomic_load(src + ((size_t)sg * nb + b) * mpad, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
      };
      // this wave's segments: wave, wave + 4, ...
      for (int sg0 = wave; sg0 < n_seg; sg0 += kWaves * kJ) {
        unsigned long long v[kJ][NB];
#pragma unroll
        for (int jj = 0; jj < kJ; ++jj)
#pragma unroll
          for (int b = 0; b < NB; ++b)
            if (b < nb) v[jj][b] = part(min(sg0 + kWaves * jj, n_seg - 1), b);
        for (int round = 0;; ++round) {
          bool ready = true;
#pragma unroll
          for (int jj = 0; jj < kJ; ++jj)
#pragma unroll
            for (int b = 0; b < NB; ++b)
              if (b < nb && sg0 + kWaves * jj < n_seg && (uint32_t)(v[jj][b] >> 32) != phase) {
                ready = false;
                v[jj][b] = part(sg0 + kWaves * jj, b);
              }
          if (ready) break;
          if (round >= kMaxRounds) {
            lost = true;
            break;
          }
        }
#pragma unroll
        for (int jj = 0; jj < kJ; ++jj)
#pragma unroll
          for (int b = 0; b < NB; ++b)
            if (b < nb && sg0 + kWaves * jj < n_seg) sums[b] += __uint_as_float((uint32_t)v[jj][b]);
      }
      if (lost)
#pragma unroll
        for (int b = 0; b < NB; ++b) sums[b] = __builtin_nanf("");
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (b < nb) {  // uniform over the workgroup
        __syncthreads();
        red[wave * 64 + lane] = sums[b];
        __syncthreads();
        if (wave == 0 && live) {
          const float t = ((red[lane] + red[64 + lane]) + red[128 + lane]) + red[192 + lane];
          ka->y[(size_t)b * rows + m] = __half_as_ushort(__float2half_rn(t));
        }
      }
    }
  }
  // every workgroup of the stripe has published (so has read the phase) by
  // the time a reducer gets here, and the next call starts after this kernel
  // ends: advance the tag (0 is skipped, the workspace's initial contents).
  // A reducer still gathering keeps its own copy of the phase.
  if (jr == n_red - 1 && threadIdx.x == 0) ka->phase[r] = phase + 1 == 0 ? 1u : phase + 1;
}

using spdp::fail;

int hip_fail(hipError_t e, const char* what) {
  return fail(SPDP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Split-K heuristic: about 7168 waves (one full load of the 256 CUs at seven
// workgroups each, so that early finishers are replaced), at most kMaxSegments
// segments per stripe (the gather then needs one round of loads), every wave
// covering a multiple of 16 columns and at most kMaxWaveCols of them.
// SPDP_SPLITK overrides the number of segments (for tuning).
constexpr int64_t kTargetWaves = 7168;
constexpr int64_t kMaxSegments = 48;
void choose_split(const spdp_matrix* m, int* segments, int* wave_cols) {
  const int64_t cols = m->cols;
  const int64_t stripes = std::max<int64_t>(1, m->n_stripes);
  int64_t want = std::min<int64_t>(kMaxSegments,
                                   std::max<int64_t>(1, (kTargetWaves + kWaves * stripes - 1) / (kWaves * stripes)));
  if (const char* env = std::getenv("SPDP_SPLITK")) {
    const long v = std::strtol(env, nullptr, 10);
    if (v >= 1) want = v;
  }
  const int64_t min_seg = (cols + kWaves * kMaxWaveCols - 1) / (kWaves * kMaxWaveCols);
  const int64_t max_seg = std::max<int64_t>(1, (cols + kWaves * 16 - 1) / (kWaves * 16));
  const int64_t s = std::max(min_seg, std::min(want, max_seg));
  int64_t wc = (cols + s * kWaves - 1) / (s * kWaves);
  wc = std::min<int64_t>(kMaxWaveCols, (wc + 15) / 16 * 16);
  *wave_cols = (int)wc;
  *segments = (int)((cols + wc * kWaves - 1) / (wc * kWaves));
}

// The workspace holds {fp32, phase} pairs for all segments; it
// starts zeroed and phases are never 0, so nothing in it matches a call
// before that call has written it.
int ensure_workspace(spdp_matrix* m, int batch, int segments) {
  const size_t need = (size_t)segments * batch * m->n_stripes * m->tile_m;
  if (need <= m->partial_floats) return SPDP_OK;
  if (m->d_partials) {
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    (void)hipFree(m->d_partials);
    m->d_partials = nullptr;
    m->partial_floats = 0;
  }
  hipError_t e = hipMalloc(&m->d_partials, need * sizeof(unsigned long long));
  if (e != hipSuccess) {
    m->d_partials = nullptr;
    return e == hipErrorOutOfMemory ? fail(SPDP_ERR_OOM, "hipMalloc of the split-K workspace failed")
                                    : hip_fail(e, "hipMalloc");
  }
  e = hipMemset(m->d_partials, 0, need * sizeof(unsigned long long));
  if (e != hipSuccess) return hip_fail(e, "hipMemset");
  e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  m->partial_floats = need;
  return SPDP_OK;
}

void release_device(spdp_matrix* m) {
  if (m->device < 0) return;
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(m->device);
  (void)hipDeviceSynchronize();
  void* ptrs[] = {m->d_tile_offset, m->d_col_info, m->d_bitmap, m->d_values, m->d_partials, m->d_phase};
  for (void* p : ptrs)
    if (p) (void)hipFree(p);
  m->d_tile_offset = m->d_col_info = m->d_bitmap = m->d_values = nullptr;
  m->d_partials = nullptr;
  m->d_phase = nullptr;
  m->partial_floats = 0;
  if (prev >= 0) (void)hipSetDevice(prev);
}

// Every device array gets kTailBytes of zeroed slack after its last element so
// that the kernel's fixed-width scalar loads (all four bitmap words of a
// column, whatever tile_m is) never leave the allocation.
constexpr size_t kTailBytes = 256;

template <class T>
int upload(const std::vector<T>& v, void** dst) {
  const size_t bytes = v.size() * sizeof(T) + kTailBytes;
  hipError_t e = hipMalloc(dst, bytes);
  if (e != hipSuccess) {
    *dst = nullptr;
    return e == hipErrorOutOfMemory ? fail(SPDP_ERR_OOM, "hipMalloc of the format arrays failed")
                                    : hip_fail(e, "hipMalloc");
  }
  e = hipMemset(static_cast<char*>(*dst) + v.size() * sizeof(T), 0, kTailBytes);
  if (e != hipSuccess) return hip_fail(e, "hipMemset");
  if (!v.empty()) {
    e = hipMemcpy(*dst, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
  }
  return SPDP_OK;
}

template <int NB, int WPC>
hipError_t launch_one(const KernelArgs& args, dim3 grid, hipStream_t stream) {
  hipLaunchKernelGGL((spmspv_kernel<NB, WPC>), grid, dim3(kThreads), 0, stream, args);
  return hipGetLastError();
}

template <int NB>
hipError_t launch(const KernelArgs& args, int wpc, dim3 grid, hipStream_t stream) {
  switch (wpc) {
    case 1: return launch_one<NB, 1>(args, grid, stream);
    case 2: return launch_one<NB, 2>(args, grid, stream);
    case 3: return launch_one<NB, 3>(args, grid, stream);
    default: return launch_one<NB, 4>(args, grid, stream);
  }
}

}  // namespace

extern "C" {

int spdp_encode(const uint16_t* W, int64_t rows, int64_t cols, int32_t tile_m,
                int32_t tile_k, spdp_handle_t* out) {
  spdp::clear_error();
  if (!out) return fail(SPDP_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  spdp_matrix* m = new (std::nothrow) spdp_matrix();
  if (!m) return fail(SPDP_ERR_OOM, "host allocation failed");
  int st = spdp::encode_host_arrays(W, rows, cols, tile_m, tile_k, m);
  if (st != SPDP_OK) {
    delete m;
    return st;
  }
  // the kernel packs a GTile column index (the all-zero padding column
  // included) into 26 bits and addresses values and bitmaps with 32-bit
  // byte offsets
  if (m->n_gtiles * m->tile_k + 1 >= (int64_t(1) << 26)) {
    delete m;
    return fail(SPDP_ERR_UNSUPPORTED, "more than 2^26 - 2 GTile columns (row stripes x padded columns)");
  }
  if ((uint64_t)m->values.size() * 2 + kTailBytes >= (uint64_t(1) << 32)) {
    delete m;
    return fail(SPDP_ERR_UNSUPPORTED, "more than 4 GiB of padded values");
  }
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    delete m;
    return hip_fail(e, "hipGetDevice");
  }
  m->device = dev;
  st = upload(m->tile_offset, &m->d_tile_offset);
  if (st == SPDP_OK) st = upload(m->col_info, &m->d_col_info);
  if (st == SPDP_OK) st = upload(m->bitmap, &m->d_bitmap);
  if (st == SPDP_OK) st = upload(m->values, &m->d_values);
  if (st == SPDP_OK) {
    // every stripe starts in phase 1
    std::vector<uint32_t> ones((size_t)m->n_stripes, 1u);
    e = hipMalloc(&m->d_phase, ones.size() * sizeof(uint32_t));
    if (e != hipSuccess) {
      m->d_phase = nullptr;
      st = hip_fail(e, "hipMalloc");
    } else {
      e = hipMemcpy(m->d_phase, ones.data(), ones.size() * sizeof(uint32_t), hipMemcpyHostToDevice);
      if (e != hipSuccess) st = hip_fail(e, "hipMemcpy");
    }
  }
  if (st == SPDP_OK) {
    int segments = 1, wave_cols = 16;
    choose_split(m, &segments, &wave_cols);
    st = ensure_workspace(m, 1, segments);
  }
  if (st != SPDP_OK) {
    release_device(m);
    delete m;
    return st;
  }
  *out = m;
  return SPDP_OK;
}

int spdp_reserve(spdp_handle_t h, int32_t max_batch) {
  spdp::clear_error();
  if (!h) return fail(SPDP_ERR_INVALID_ARG, "handle is NULL");
  if (h->device < 0) return fail(SPDP_ERR_INVALID_ARG, "handle has no device copy");
  if (max_batch < 1 || max_batch > kMaxBatch)
    return fail(SPDP_ERR_INVALID_ARG, "max_batch must lie in [1, 32]");
  int segments = 1, wave_cols = 16;
  choose_split(h, &segments, &wave_cols);
  return ensure_workspace(h, max_batch, segments);
}

int spdp_spmspv(spdp_handle_t h, const uint16_t* X, int32_t batch, float threshold,
                uint16_t* Y, void* stream) {
  spdp::clear_error();
  if (!h) return fail(SPDP_ERR_INVALID_ARG, "handle is NULL");
  if (h->device < 0) return fail(SPDP_ERR_INVALID_ARG, "handle has no device copy");
  if (!X || !Y) return fail(SPDP_ERR_INVALID_ARG, "X or Y is NULL");
  if (batch < 1 || batch > kMaxBatch) return fail(SPDP_ERR_INVALID_ARG, "batch must lie in [1, 32]");
  if ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(Y)) & 15)
    return fail(SPDP_ERR_INVALID_ARG, "X and Y must be 16-byte aligned");
  {
    const uintptr_t x0 = reinterpret_cast<uintptr_t>(X);
    const uintptr_t x1 = x0 + (uintptr_t)batch * h->cols * 2;
    const uintptr_t y0 = reinterpret_cast<uintptr_t>(Y);
    const uintptr_t y1 = y0 + (uintptr_t)batch * h->rows * 2;
    if (x0 < y1 && y0 < x1) return fail(SPDP_ERR_INVALID_ARG, "X and Y overlap");
  }
  int32_t code = 0;
  int st = spdp_threshold_code(threshold, &code);
  if (st != SPDP_OK) return st;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != h->device) return fail(SPDP_ERR_INVALID_ARG, "current device differs from the handle's");

  int segments = 1, wave_cols = 16;
  choose_split(h, &segments, &wave_cols);
  st = ensure_workspace(h, batch, segments);
  if (st != SPDP_OK) return st;

  KernelArgs args;
  args.tile_offset = static_cast<const uint32_t*>(h->d_tile_offset);
  args.col_info = static_cast<const uint32_t*>(h->d_col_info);
  args.bitmap = static_cast<const uint64_t*>(h->d_bitmap);
  args.values = static_cast<const uint16_t*>(h->d_values);
  args.x = X;
  args.y = Y;
  args.partials = h->d_partials;
  args.phase = h->d_phase;
  args.rows = (int)h->rows;
  args.cols = (int)h->cols;
  args.tile_m = h->tile_m;
  const int wpc = h->tile_m / 64;
  args.zero_col = (uint32_t)(h->n_gtiles * h->tile_k);
  args.tk_log2 = __builtin_ctz((unsigned)h->tile_k);
  args.n_colblocks = (int)h->n_colblocks;
  args.n_stripes = (int)h->n_stripes;
  args.batch = batch;
  args.code = code;
  args.wave_cols = wave_cols;
  args.segments = segments;

  const dim3 grid((unsigned)segments, (unsigned)h->n_stripes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (batch <= 1)
    e = launch<1>(args, wpc, grid, s);
  else if (batch <= 2)
    e = launch<2>(args, wpc, grid, s);
  else if (batch <= 4)
    e = launch<4>(args, wpc, grid, s);
  else if (batch <= 8)
    e = launch<8>(args, wpc, grid, s);
  else if (batch <= 16)
    e = launch<16>(args, wpc, grid, s);
  else
    e = launch<32>(args, wpc, grid, s);
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return SPDP_OK;
}

void spdp_free(spdp_handle_t h) {
  if (!h) return;
  release_device(h);
  delete h;
}

}  // extern "C"
