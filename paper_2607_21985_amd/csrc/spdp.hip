// Device side of libspdp for gfx950 (MI355X): the fused decode-time spMspV
// kernel over Tiled-CBC weights (Sec. 4.2) and the C-ABI entry points that
// own device memory.
//
// One launch runs one or several independent products (a decoder's q, k and
// v, or gate and up, read one input); each product is a grid row of
// workgroups, one per (row stripe, K segment). A workgroup does the whole
// path for its piece:
//   1. activity: each wave reads a K range of the activations and takes the
//      strict magnitude test |x| > t as an integer compare on fp16 bits;
//      64-lane ballots (union over the batch) and mbcnt positions compact the
//      workgroup's active columns into one list in LDS (Sec. 4.2, XTile
//      loading and the activation-aware selection of GTile loading); ColInfo
//      and TileOffset of the range arrive in the same round trip as the
//      activations;
//   2. data (Sec. 4.2.2, metadata first, data second): the list is cut into
//      batches of four columns, spread evenly over the four waves; each wave
//      streams its batches through a two-slot ring in LDS with global->LDS
//      DMA (16-byte loads of the padded values, two columns per instruction,
//      plus the batch's bitmap words), so loads in flight hold no registers;
//      on small one-token products each wave first requests a batch of its
//      own first active columns, before the list is built;
//   3. bitmap decode (HAD-SMBD, Sec. 4.2.1): the bitmap words come from
//      scalar loads (their lines are in L2 once the batch's DMA has landed);
//      lane i of word w reads its value at the word's masked popcount below
//      bit i (v_mbcnt_lo/hi, the paper's MaskedPopcount) plus the popcount of
//      the column's earlier words;
//   4. accumulate in fp32 on the vector ALUs with fp16 operands: one or two
//      tokens, v_fma_mix under EXEC = the bitmap word (rows without a nonzero
//      do nothing); more tokens, the two columns of a pair selected into the
//      halves of one register and one v_dot2_f32_f16 per token; no matrix
//      cores (Sec. 3.3 challenge 2, Sec. 4.2 step 5);
//   5. split-K (Sec. 4.2.3): each workgroup reduces its 4 waves in LDS and
//      stores its fp32 partial sums to the product's workspace, each value
//      paired with the stripe's phase number in one 8-byte store; the
//      stripe's last segments gather the partials until every one carries
//      the current phase, add them in a fixed order, write fp16 Y (round to
//      nearest even), and the first of them advances the stripe's phase for
//      the next call. No
//      counter, no fence, no host-side state: a partial is usable as soon as
//      its own store has landed, and a captured graph replays correctly.
// With low-bit Values (spdp_encode_rtn, Sec. 5.1's quantization setup) the
// same kernel reads one-byte codes: step 2 streams 16 codes per 16-byte
// chunk, step 3 addresses bytes and turns each code into an fp16 integer
// (exact), steps 4-5 are unchanged, and the row's scale multiplies the
// gathered sum once before the fp16 rounding.

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "internal.h"

namespace {

constexpr int kWaves = 4;                 // waves per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxWords = 4;              // tile_m <= 256: at most 4 bitmap words per column
constexpr int kSlotBytes = 64 * kMaxWords * 2;  // LDS slot: one column of one stripe (fp16)
constexpr int kBatch = 4;                 // active columns per DMA batch (one decode quad)
constexpr int kQuad = 4;                  // columns decoded together
// Columns whose activity one wave tests per range: up to 128 (the widest
// products keep few segments). From two tokens on the kernels also come in
// a 64-column form, launched when no product of the launch has wider
// ranges: it tests one 64-column chunk per lane instead of two (the second
// is empty then), and its smaller list and activation arrays in LDS buy an
// occupancy step at 16 and 32 tokens. A range of at most 64 columns gives
// the same bits in both forms. The one-token kernel keeps the 128-column
// form (its 64-column form was 1-3 % slower on the Llama-70B layer).
constexpr int kMaxWaveCols = 128;
constexpr int kNarrowWaveCols = 64;
constexpr int kMaxBatch = 32;
constexpr int kBmBytes = kBatch * kMaxWords * 8;          // bitmap words of one batch
constexpr int kBatchBytes = kBatch * kSlotBytes + kBmBytes;  // one ring slot
constexpr int kDmaPerBatch = kBatch / 2 + 1;  // 16-byte value loads (two columns each) + one bitmap load

// One product of a launch: the matrix's device arrays, the call's input and
// output, and the matrix's split.
struct MatArgs {
  const uint32_t* tile_offset;
  const uint32_t* col_info;
  const uint64_t* bitmap;
  const uint16_t* values;  // fp16 values, or one-byte codes (the kernel's Q form)
  const float* scales;     // Q form: one scale per row
  const uint16_t* x;
  uint16_t* y;
  // [segments][batch][n_stripes * tile_m]: {fp32 bits, phase} pairs
  unsigned long long* partials;
  // the tag of this call's partials, never 0 (the workspace starts zeroed).
  // A handle's own workspace has one phase per stripe (phase_step 1,
  // epoch_done NULL): the tag is phase[r], and the stripe's first reducer
  // advances it. The library's static workspace, shared by every handle, has
  // one device-wide epoch (phase_step 0): the tag is *phase + 1 (0 skipped);
  // each stripe's first reducer counts itself in *epoch_done, and the last
  // stripe's stores the tag as the new epoch and clears the count.
  uint32_t* phase;
  uint32_t* epoch_done;
  int phase_step;
  int rows, cols;
  int tile_m, tk_log2, n_colblocks, n_stripes;
  int code;       // threshold code: active iff code < (x & 0x7fff) <= 0x7c00
  int wave_cols;  // columns per wave (multiple of 16, <= kMaxWaveCols)
  int segments;   // workgroups per row stripe
  int n_wg;       // segments * n_stripes
  uint32_t zero_col;  // column index whose bitmap lies in the zeroed tail padding
  // nonzero: each wave requests its first batch before the workgroup list is
  // built (a property of the product and the batch, never of the launch, so
  // that grouping does not change the summation order)
  int early_first;
  // with the batch's shared column set (the kernel's BMASK form): a column
  // is active iff the fp32 running sum of |x[b, k]| over the tokens exceeds
  // batch_thr = fp32(batch * t), every token's activation kept there
  float batch_thr;
  // consecutive K ranges (of kWaves x wave_cols columns) per workgroup
  int passes;
};

// A launch runs up to kMaxGroup independent products (same tile height and
// batch): grid row y serves product y, its workgroup x being stripe
// x / segments, segment x % segments (segments ascending within a stripe);
// workgroups past the product's n_wg exit at once.
constexpr int kMaxGroup = 8;
struct LaunchArgs {
  MatArgs m[kMaxGroup];
  int batch;
};

// Per-wave ring of batch slots in LDS, filled by global->LDS DMA: deep enough
// that at the Llama-7B shapes a wave's whole share is requested at once.
template <int NB>
struct Smem {
  static constexpr int kSlots = 2;
  static constexpr int kRingBytes = kWaves * kSlots * kBatchBytes;
  static constexpr int kSlice = NB < 4 ? NB : 4;  // tokens per cross-wave reduction pass
  static constexpr int kRed = kWaves * kSlice * 256 * 4;
  static_assert(kRed <= kRingBytes, "reduction reuses the ring");
};

__device__ __forceinline__ uint32_t mbcnt64(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
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

// The same for two tokens: one EXEC word, then one FMA per token (x0, x1:
// the tokens' dwords of the column's pair, the half picked by op_sel).
#define SPDP_FMA2(W, SEL) "v_fma_mix_f32 %[a" #W "0], %[v" #W "], %[x0], %[a" #W "0] " SEL "\n\t" \
                            "v_fma_mix_f32 %[a" #W "1], %[v" #W "], %[x1], %[a" #W "1] " SEL "\n\t"
#define SPDP_COLUMN2(SEL) \
  if constexpr (WPC == 1) {                                                          \
    asm volatile("s_and_saveexec_b64 %[sv], %[m0]\n\t" SPDP_FMA2(0, SEL) "s_mov_b64 exec, %[sv]" \
                 : [a00] "+v"(acc[0][0]), [a01] "+v"(acc[0][1]), [sv] "=&s"(save) \
                 : [m0] "s"(m[0]), [v0] "v"(v[0]), [x0] "v"(x0), [x1] "v"(x1) \
                 : "scc"); \
  } else if constexpr (WPC == 2) {                                                          \
    asm volatile("s_and_saveexec_b64 %[sv], %[m0]\n\t" SPDP_FMA2(0, SEL) "s_and_b64 exec, %[sv], %[m1]\n\t" SPDP_FMA2(1, SEL) "s_mov_b64 exec, %[sv]" \
                 : [a00] "+v"(acc[0][0]), [a01] "+v"(acc[0][1]), [a10] "+v"(acc[1][0]), [a11] "+v"(acc[1][1]), [sv] "=&s"(save) \
                 : [m0] "s"(m[0]), [m1] "s"(m[1]), [v0] "v"(v[0]), [v1] "v"(v[1]), [x0] "v"(x0), [x1] "v"(x1) \
                 : "scc"); \
  } else if constexpr (WPC == 3) {                                                          \
    asm volatile("s_and_saveexec_b64 %[sv], %[m0]\n\t" SPDP_FMA2(0, SEL) "s_and_b64 exec, %[sv], %[m1]\n\t" SPDP_FMA2(1, SEL) "s_and_b64 exec, %[sv], %[m2]\n\t" SPDP_FMA2(2, SEL) "s_mov_b64 exec, %[sv]" \
                 : [a00] "+v"(acc[0][0]), [a01] "+v"(acc[0][1]), [a10] "+v"(acc[1][0]), [a11] "+v"(acc[1][1]), [a20] "+v"(acc[2][0]), [a21] "+v"(acc[2][1]), [sv] "=&s"(save) \
                 : [m0] "s"(m[0]), [m1] "s"(m[1]), [m2] "s"(m[2]), [v0] "v"(v[0]), [v1] "v"(v[1]), [v2] "v"(v[2]), [x0] "v"(x0), [x1] "v"(x1) \
                 : "scc"); \
  } else if constexpr (WPC == 4) {                                                          \
    asm volatile("s_and_saveexec_b64 %[sv], %[m0]\n\t" SPDP_FMA2(0, SEL) "s_and_b64 exec, %[sv], %[m1]\n\t" SPDP_FMA2(1, SEL) "s_and_b64 exec, %[sv], %[m2]\n\t" SPDP_FMA2(2, SEL) "s_and_b64 exec, %[sv], %[m3]\n\t" SPDP_FMA2(3, SEL) "s_mov_b64 exec, %[sv]" \
                 : [a00] "+v"(acc[0][0]), [a01] "+v"(acc[0][1]), [a10] "+v"(acc[1][0]), [a11] "+v"(acc[1][1]), [a20] "+v"(acc[2][0]), [a21] "+v"(acc[2][1]), [a30] "+v"(acc[3][0]), [a31] "+v"(acc[3][1]), [sv] "=&s"(save) \
                 : [m0] "s"(m[0]), [m1] "s"(m[1]), [m2] "s"(m[2]), [m3] "s"(m[3]), [v0] "v"(v[0]), [v1] "v"(v[1]), [v2] "v"(v[2]), [v3] "v"(v[3]), [x0] "v"(x0), [x1] "v"(x1) \
                 : "scc"); \
  }
template <int WPC, bool XHI>
__device__ __forceinline__ void masked_fma_column2(float (&acc)[WPC][2], const uint32_t (&v)[WPC], uint32_t x0,
                                                   uint32_t x1, const uint64_t (&m)[WPC]) {
  uint64_t save;
  static_assert(WPC >= 1 && WPC <= 4, "at most four bitmap words per column");
  if constexpr (XHI) {
    SPDP_COLUMN2("op_sel:[0,1,0] op_sel_hi:[1,1,0]")
  } else {
    SPDP_COLUMN2("op_sel_hi:[1,1,0]")
  }
}
#undef SPDP_COLUMN2
#undef SPDP_FMA2



// {a where word ma has the lane's bit, else 0} | {b likewise under mb} << 16,
// for a and b zero-extended fp16 bits: two selects that each write one half
// of the result (SDWA, the other half kept), the words as VCC.
__device__ __forceinline__ uint32_t pair_under_words(uint32_t a, uint32_t b, uint64_t ma, uint64_t mb) {
  uint32_t p;
  asm("s_mov_b64 vcc, %[ma]\n\t"
      "v_cndmask_b32_sdwa %[p], 0, %[a], vcc dst_sel:WORD_0 dst_unused:UNUSED_PRESERVE src0_sel:DWORD src1_sel:WORD_0\n\t"
      "s_mov_b64 vcc, %[mb]\n\t"
      "v_cndmask_b32_sdwa %[p], 0, %[b], vcc dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:DWORD src1_sel:WORD_0"
      : [p] "=&v"(p)
      : [a] "v"(a), [b] "v"(b), [ma] "s"(ma), [mb] "s"(mb)
      : "vcc");
  return p;
}

// The same pair for a matrix-core operand. The compiler's hazard checks do
// not look inside the assembly: an MFMA that reads a VGPR a VALU
// instruction has just written needs wait states between them, so two
// follow the selects (a GPU test failed on the rows of a batch's last word,
// whose MFMA came one wait state after its select).
__device__ __forceinline__ uint32_t pair_under_words_mfma(uint32_t a, uint32_t b, uint64_t ma, uint64_t mb) {
  uint32_t p;
  asm("s_mov_b64 vcc, %[ma]\n\t"
      "v_cndmask_b32_sdwa %[p], 0, %[a], vcc dst_sel:WORD_0 dst_unused:UNUSED_PRESERVE src0_sel:DWORD src1_sel:WORD_0\n\t"
      "s_mov_b64 vcc, %[mb]\n\t"
      "v_cndmask_b32_sdwa %[p], 0, %[b], vcc dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:DWORD src1_sel:WORD_0\n\t"
      "s_nop 1"
      : [p] "=&v"(p)
      : [a] "v"(a), [b] "v"(b), [ma] "s"(ma), [mb] "s"(mb)
      : "vcc");
  return p;
}


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

// Global -> LDS DMA of 16 (or 4) bytes per lane from base + off: lane l's
// bytes land at lds + 16 l (4 l); lanes outside EXEC write nothing. Issued
// as assembly so that the compiler does not order every later LDS read
// behind all outstanding DMA (the loads target ring slots that the reads
// below do not touch); the waits for them are explicit.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// The compiler's hazard checks do not look inside inline assembly: a vector
// memory instruction needs 5 wait states after a VALU instruction writes an
// SGPR it reads (the compiler may have just restored the base pointer from a
// VGPR lane with v_readlane) and 1 after an M0 write, so each load is
// preceded by s_nop 4.
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

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float float16_t __attribute__((ext_vector_type(16)));
typedef float float4_t __attribute__((ext_vector_type(4)));
// MFMA form: a wave's dense tile of decoded weights, one row per matrix row
// of the stripe, 8 columns (two batches) per row, padded to 24 bytes
constexpr int kMRowBytes = 24;

// NB: tokens per call rounded up to a power of two; WPC: bitmap words per
// column (tile_m / 64); Q: Values are one-byte round-to-nearest codes with a
// scale per row (else fp16); MM: accumulate on the matrix cores (8 or more
// tokens: the product of a batch of 8 active columns with up to 32 tokens
// is a small dense contraction; see step 4).
template <int NB, int WPC, bool EARLY, bool BMASK, bool Q, bool MM, bool MP, int MWC>
__device__ __forceinline__ void spmspv_body() {
  static_assert(!MM || (NB >= 8 && !Q && !EARLY), "the MFMA form serves 8 or more tokens of fp16 values");
  static_assert(!MP || (NB >= 4 && !Q && !EARLY), "several K ranges: 3 or more tokens of fp16 values");
  static_assert(MWC == kNarrowWaveCols || MWC == kMaxWaveCols, "64- or 128-column ranges");
  // the workgroup's list capacity; with early first batches the list holds
  // at most kWgCols - kWaves kBatch columns (each wave's first kBatch active
  // columns form its own first batch) plus the last batch's padding, and
  // the waves' first batches follow it at kFirst; without, the list may use
  // every entry
  constexpr int kWgCols = kWaves * MWC;
  constexpr int kFirst = kWgCols - kWaves * kBatch + kBatch;
  static_assert(kFirst % kBatch == 0 && kFirst + kWaves * kBatch == kWgCols + kBatch, "list layout");
  using S = Smem<NB>;
  constexpr int kSlots = S::kSlots;
  __shared__ __attribute__((aligned(1024))) unsigned char ring[S::kRingBytes];
  __shared__ __attribute__((aligned(16))) unsigned char mt_s[MM ? kWaves * 64 * WPC * kMRowBytes : 16];
  // the workgroup's active columns in activity order: {byte offset of the
  // column's values, the column's bitmap offset and the index of its
  // last 16-byte chunk}; padded to a whole batch with entries that load
  // nothing of use
  __shared__ uint2 ent_s[kWgCols + kBatch];
  // the entries' masked activations: per pair of entries a row of NB dwords
  // (token b: entry 2j in the low half, 2j + 1 in the high), from four
  // tokens on padded by one dword so that consecutive pairs start in
  // different banks; the MFMA form keeps each entry's NB values together
  constexpr int kXRow = (MM || NB < 4) ? NB : NB + 1;
  // from four tokens (vector forms) the pair rows of a quad are interleaved
  // by token, so that the 4x4x4 product's A operand (both pair rows of one
  // token) is one 8-byte read: dword (q kXRow + b) 2 + h holds token b of
  // entries 4q + 2h (low half) and 4q + 2h + 1 (high half); the row of
  // kXRow = NB + 1 keeps the quads' stores in different banks
  constexpr bool kQuadRows = !MM && NB >= 4;
  auto xs_at = [&](int p, int b) __attribute__((always_inline)) {
    return kQuadRows ? (((p >> 2) * kXRow + b) * 2 + ((p >> 1) & 1)) * 2 + (p & 1)
                     : ((p >> 1) * kXRow + b) * 2 + (p & 1);
  };
  __shared__ __attribute__((aligned(16))) uint16_t xs_s[(kWgCols + kBatch) * kXRow];
  __shared__ int cnt_s[kWaves];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the product this workgroup serves, and its (stripe, segment)
  const const_ptr<LaunchArgs> L = reload_args<LaunchArgs>();
  const int mi = blockIdx.y;
  const const_ptr<MatArgs> A = &L->m[mi];
  // every field this prologue needs is requested before the first test, so
  // that the kernel-argument reads form one round trip
  const uint32_t local = blockIdx.x;
  const uint32_t n_wg = (uint32_t)A->n_wg;
  const uint32_t n_seg0 = (uint32_t)A->segments;
  const int batch = L->batch;
  const int early_first = EARLY ? A->early_first : 0;
  const float batch_thr = BMASK ? A->batch_thr : 0.0f;
  const int tk_log2 = A->tk_log2;
  const int n_colblocks = A->n_colblocks;
  const int code = A->code;
  const int cols = A->cols;
  const int wave_cols = A->wave_cols;
  const uint32_t* const phase_p = A->phase;
  const uint32_t* const col_info_p = A->col_info;
  const uint32_t* const tile_offset_p = A->tile_offset;
  const uint16_t* const x_p = A->x;
  const void* const values = A->values;
  const void* const bitmap = A->bitmap;
  const uint32_t zero_col = A->zero_col;
  asm volatile("" ::"s"(n_seg0), "s"(batch), "s"(tk_log2), "s"(n_colblocks), "s"(code), "s"(cols),
               "s"(wave_cols), "s"(phase_p), "s"(col_info_p), "s"(tile_offset_p), "s"(x_p), "s"(values),
               "s"(bitmap), "s"(zero_col), "s"(early_first), "s"(batch_thr));
  if (local >= n_wg) return;  // the whole workgroup: no barrier has been reached
  const int r = (int)(local / n_seg0);
  const int seg = (int)(local - (uint32_t)r * n_seg0);
  const int tk_mask = (1 << tk_log2) - 1;
  const int g_row = r * n_colblocks;

  float acc[WPC][NB];
#pragma unroll
  for (int w = 0; w < WPC; ++w)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[w][b] = 0.0f;
  // from four tokens on (vector-ALU kernels): word w's rows x tokens 4g ..
  // 4g + 3, lane = row, in the 4x4x4 MFMA's accumulator layout
  constexpr bool kM4 = !MM && NB >= 4;
  float4_t acc4[kM4 ? WPC : 1][kM4 ? NB / 4 : 1];
#pragma unroll
  for (int w = 0; w < (kM4 ? WPC : 1); ++w)
#pragma unroll
    for (int g = 0; g < (kM4 ? NB / 4 : 1); ++g) acc4[w][g] = float4_t{0.0f, 0.0f, 0.0f, 0.0f};
  // MFMA form: the stripe's 32-row blocks x 32 tokens (tokens past the
  // batch stay 0), in the 32x32 accumulator layout
  constexpr int kMBlocks = 2 * WPC;
  float16_t macc[MM ? kMBlocks : 1];
#pragma unroll
  for (int i = 0; i < (MM ? kMBlocks : 1); ++i) macc[i] = float16_t{};

  // The workgroup walks `passes` consecutive K ranges (one unless the batch
  // and the product are large: fewer segments then mean fewer split-K
  // partials, whose bytes grow with the batch), accumulating into the same
  // registers; each pass tests its range, builds its list and streams it.
  // The stripe's phase is read in the first pass. Only the MP kernels have
  // the loop (in the others it costs 3-6 % at one pass).
  const int passes = MP ? A->passes : 1;
  uint32_t phase = 0;
  for (int pass = 0; pass < passes; ++pass) {
    if (pass > 0) __syncthreads();  // the last pass's list, activations and ring are free
    // in the several-range kernels the batch, the column count, X's address
    // and the threshold code pass through an empty asm per pass, so that what
    // the prologue derives from them per token (row offsets, lane masks) is
    // computed where it is used instead of being hoisted out of the pass
    // loop, where it would hold scalar registers through every pass
    int batch_q = batch, cols_q = cols, code_q = code;
    const uint16_t* x_q = x_p;
    if constexpr (MP) asm volatile("" : "+s"(batch_q), "+s"(cols_q), "+s"(x_q), "+s"(code_q));
    const int k_begin = ((seg * passes + pass) * kWaves + wave) * wave_cols;
    const int range = max(0, min(wave_cols, cols - k_begin));

    // ---- 1. each wave's K range: activations and column metadata in one round
    // trip (ColInfo/TileOffset are fetched for every column of the range, which
    // removes a dependent memory round trip; their cache lines are shared by
    // neighbouring columns, so little extra traffic results).
    // All loads are unconditional so that they leave back to back and are
    // waited for once: lanes past the range (and waves past the last column)
    // read column k_begin's or column 0's entries, tokens past the batch read
    // the last token; none of those is used below.
    constexpr int kChunks = MWC / 64;
    uint32_t ci[kChunks], to[kChunks], colx[kChunks], xb[kChunks][NB];
    const int k_safe = k_begin < cols ? k_begin : 0;
  #pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int off = 64 * c + lane;
      const int k = off < range ? k_begin + off : k_safe;
      const int g = g_row + (k >> tk_log2);
      colx[c] = ((uint32_t)g << tk_log2) + (uint32_t)(k & tk_mask);
      ci[c] = col_info_p[colx[c]];
      to[c] = tile_offset_p[g];
  #pragma unroll
      for (int b = 0; b < NB; ++b) xb[c][b] = x_q[(size_t)min(b, batch_q - 1) * cols_q + k];
    }
    // the stripe's phase: written by the previous call's last segment, read
    // by every workgroup of the stripe before any of them publishes (the
    // kernel boundary makes the write visible, so an ordinary cached load
    // serves). A vector load issued after the loads above, so that waiting for
    // them does not wait for it (loads return in order), waited for after the
    // list is built; a scalar load would share the LDS wait counter, and the
    // compiler would wait for it at the first LDS barrier.
    uint32_t phase_lane = 0;
    if (pass == 0)
      phase_lane = __hip_atomic_load(phase_p + r * A->phase_step, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    // activity: the union of the tokens' sets, or the batch's shared set.
    // From four tokens on the activations are also masked here, once per
    // column (one compare per token gives both the token's bit and its
    // masked value, so no per-token mask stays live in scalar registers): xm
    // holds them two tokens to a dword (zero outside the token's set and past
    // the batch), the registers the list entry is written from.
    uint64_t actm[kChunks];
    constexpr bool kXm = MM || NB >= 4;
    uint32_t xm[kChunks][kXm ? NB / 2 : 1];
    int n_w = 0;
  #pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const bool in = 64 * c + lane < range;
      uint64_t act = 0;
      if constexpr (kXm) {
        // mag in (code, 0x7C00] is one unsigned compare for code in [-1, 0x7C00]
        const uint32_t lo = (uint32_t)(code_q + 1), span = (uint32_t)(0x7C00 - code_q);
        uint64_t any = 0;
  #pragma unroll
        for (int j = 0; j < NB / 2; ++j) {
          uint32_t h[2];
  #pragma unroll
          for (int s = 0; s < 2; ++s) {
            const int b = 2 * j + s;
            const bool on = b < batch_q && (BMASK || (xb[c][b] & 0x7FFFu) - lo < span);
            if constexpr (!BMASK) any |= __builtin_amdgcn_ballot_w64(on);
            h[s] = on ? xb[c][b] : 0u;
          }
          xm[c][j] = h[0] | (h[1] << 16);
        }
        act = any & __builtin_amdgcn_ballot_w64(in);
      }
      if constexpr (BMASK) {
        // fp32 running sum of |x| over the tokens in ascending order (NaN
        // makes it NaN, never active)
        float score = 0.0f;
  #pragma unroll
        for (int b = 0; b < NB; ++b)
          if (b < batch_q) score += __half2float(__ushort_as_half((unsigned short)(xb[c][b] & 0x7FFFu)));
        act = __builtin_amdgcn_ballot_w64(in && score > batch_thr);
      } else if constexpr (!kXm) {
  #pragma unroll
        for (int b = 0; b < NB; ++b) {
          const int mag = (int)(xb[c][b] & 0x7FFFu);
          act |= __builtin_amdgcn_ballot_w64(in && b < batch_q && mag > code_q && mag <= 0x7C00);
        }
      }
      actm[c] = act;
      n_w += __builtin_popcountll(act);
    }
    // list entry p of this lane's column of chunk c, with its masked
    // activations (every token's under the batch's shared set; pair-
    // interleaved: entries 2j and 2j+1 share a dword per token); entries of
    // the all-zero column pad a batch: they read the
    // bitmap array's zeroed tail and the first 16 bytes of the values, and
    // decode to nothing
    // An entry's second word: with tile_m a power of two (WPC 1, 2 or 4) the
    // byte offset of the column's bitmap words, a multiple of WPC x 8, with
    // the index of the column's last 16-byte chunk (< WPC x 8) in its low
    // bits, so that both come out with one AND each; with 192-row tiles the
    // column index << 6 and the chunk index.
    constexpr bool kPow2 = (WPC & (WPC - 1)) == 0;
    constexpr uint32_t kLow = kPow2 ? WPC * 8u - 1u : 63u;
    auto ent_col = [&](uint32_t col, uint32_t chunk) __attribute__((always_inline)) {
      return kPow2 ? col * (WPC * 8u) + chunk : (col << 6) | chunk;
    };
    auto ent_chunk = [&](uint32_t y) __attribute__((always_inline)) { return y & kLow; };
    auto ent_bitmap = [&](uint32_t y) __attribute__((always_inline)) {
      return kPow2 ? y & ~kLow : (y >> 6) * (WPC * 8u);
    };
    // The MFMA form keeps an entry's NB activations together (NB / 8 pieces
    // of 16 bytes, one wide store each); piece k sits at k ^ mm_swz(p), so
    // that the eight lanes of a 16-byte store phase (consecutive entries)
    // cover all 32 banks.
    constexpr int kPieces = MM ? NB / 8 : 1;
    auto mm_swz = [&](uint32_t p) __attribute__((always_inline)) {
      return (p / (8u / kPieces)) & (uint32_t)(kPieces - 1);
    };
    auto put = [&](int c, int p) __attribute__((always_inline)) {
      // 16-byte chunks of the column's padded values (8 fp16 or 16 codes each)
      const uint32_t chunks = Q ? ((ci[c] & 0xFFFFu) + 15u) >> 4 : ((ci[c] & 0xFFFFu) + 7u) >> 3;
      ent_s[p] = make_uint2((Q ? 1u : 2u) * (to[c] + (ci[c] >> 16)), ent_col(colx[c], chunks ? chunks - 1u : 0u));
      if constexpr (MM) {
        const uint32_t swz = mm_swz((uint32_t)p);
  #pragma unroll
        for (int k = 0; k < kPieces; ++k)
          *reinterpret_cast<uint4*>(&xs_s[p * NB + 8 * (k ^ swz)]) =
              make_uint4(xm[c][4 * k], xm[c][4 * k + 1], xm[c][4 * k + 2], xm[c][4 * k + 3]);
      } else {
  #pragma unroll
        for (int b = 0; b < NB; ++b) {
          if constexpr (kXm) {
            const uint32_t v = xm[c][b >> 1];
            xs_s[xs_at(p, b)] = (b & 1) ? (uint16_t)(v >> 16) : (uint16_t)v;
          } else {
            const int mag = (int)(xb[c][b] & 0x7FFFu);
            const bool on = b < batch_q && (BMASK || (mag > code_q && mag <= 0x7C00));
            xs_s[xs_at(p, b)] = on ? (uint16_t)xb[c][b] : (uint16_t)0;
          }
        }
      }
    };
    auto put_zero = [&](int p) __attribute__((always_inline)) {
      ent_s[p] = make_uint2(0u, ent_col(zero_col, 0u));
      if constexpr (MM) {
  #pragma unroll
        for (int k = 0; k < kPieces; ++k) *reinterpret_cast<uint4*>(&xs_s[p * NB + 8 * k]) = make_uint4(0u, 0u, 0u, 0u);
      } else {
  #pragma unroll
        for (int b = 0; b < NB; ++b) xs_s[xs_at(p, b)] = 0;
      }
    };

    // A batch = kBatch list entries, streamed through the wave's ring of kSlots
    // batch slots in LDS (LDS DMA, no registers held by loads in flight).
    // Values: lane l of load pr brings 16 bytes of column 2pr + (l >= 32),
    // chunk l & 31, to that column's 512-byte slot; lanes past a column's end
    // re-read its last chunk (a line the column loads anyway). Bitmaps: lane l
    // < 16 WPC brings dword l of the batch's words (column l / (2 WPC)).
    const int hsel = lane >> 5;
    const int q = lane & 31;
    unsigned char* my_ring = ring + wave * (kSlots * kBatchBytes);
    auto issue_at = [&](int e0, int si) __attribute__((always_inline)) {
      const uint32_t slot = (uint32_t)__builtin_amdgcn_readfirstlane(
          (int)lds_addr(my_ring + si * kBatchBytes));
      // the batch's entries are read before the first load is issued, so
      // that they take one LDS round trip (a load's asm orders every later
      // LDS read behind it: one round trip per load otherwise)
      uint2 ev[kBatch / 2];
  #pragma unroll
      for (int pr = 0; pr < kBatch / 2; ++pr) ev[pr] = ent_s[e0 + 2 * pr + hsel];
      const uint32_t eb = ent_s[e0 + min(lane / (2 * WPC), kBatch - 1)].y;
  #pragma unroll
      for (int pr = 0; pr < kBatch / 2; ++pr)
        dma16(values, ev[pr].x + (min((uint32_t)q, ent_chunk(ev[pr].y)) << 4), slot + pr * 2 * kSlotBytes);
      if (lane < 2 * WPC * kBatch)
        dma4(bitmap, ent_bitmap(eb) + 4u * (uint32_t)(lane % (2 * WPC)), slot + kBatch * kSlotBytes);
    };

    // ---- 2a. (when the launch asks for it) the wave's first batch: its own
    // first kBatch active columns, listed at the tail of the list arrays and
    // requested at once, so that their loads are in flight while the
    // workgroup builds its list (two barriers) from the remaining columns. The phase load has landed with
    // the loads above (loads return in order); it is read here because it is
    // the only vector load the compiler tracks and must be complete before the
    // first DMA: the compiler does not see those loads, so a wait it placed
    // for a load of its own among them would count them and drain the ring.
    // the static workspace's epoch starts at 0 (static storage), the value
    // its zeroed partials carry: a call's tag is the stored epoch plus one
    // (0 skipped), and the call stores its tag back when it is done
    if (pass == 0) {
      phase = (uint32_t)__builtin_amdgcn_readfirstlane((int)phase_lane);
      if (A->phase_step == 0) phase = phase + 1u == 0u ? 1u : phase + 1u;
    }
    asm volatile("" ::"s"(phase));
    const bool has_first = EARLY && early_first && n_w > 0;
    const int e_first = kFirst + kBatch * wave;
    if (has_first) {
      int rank0 = 0;
  #pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        if ((actm[c] >> lane) & 1) {
          const int rk = rank0 + (int)mbcnt64(actm[c]);
          if (rk < kBatch) put(c, e_first + rk);
        }
        rank0 += __builtin_popcountll(actm[c]);
      }
      if (lane >= n_w && lane < kBatch) put_zero(e_first + lane);
      issue_at(e_first, 0);
    }

    // ---- 2b. the workgroup-wide list of the remaining active columns: each
    // wave's follow those of the lower waves
    const int n_skip = EARLY && has_first ? kBatch : 0;  // ranks already in the first batch
    if (lane == 0) cnt_s[wave] = max(n_w - n_skip, 0);
    __syncthreads();
    int total = 0, pos = 0;
  #pragma unroll
    for (int v = 0; v < kWaves; ++v) {
      const int cv = cnt_s[v];
      pos += v < wave ? cv : 0;
      total += cv;
    }
    {
      int rank0 = 0;
  #pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        if ((actm[c] >> lane) & 1) {
          const int rk = rank0 + (int)mbcnt64(actm[c]);
          if (rk >= n_skip) put(c, pos + rk - n_skip);
        }
        rank0 += __builtin_popcountll(actm[c]);
      }
    }
    // pad the list's last batch
    if (wave == 0 && lane < ((kBatch - (total & (kBatch - 1))) & (kBatch - 1))) put_zero(total + lane);
    __syncthreads();

    // ---- 2c. the list's batches are split evenly over the waves; each wave
    // streams its first batch, then its share, and decodes a batch as soon as
    // its loads have landed.
    const int n_bt = (total + kBatch - 1) / kBatch;
    const int bb0 = n_bt * wave / kWaves;
    const int n_first = EARLY && has_first ? 1 : 0;
    const int n_mine = n_bt * (wave + 1) / kWaves - bb0 + n_first;
    auto entry0 = [&](int i) { return n_first && i == 0 ? e_first : (bb0 + i - n_first) * kBatch; };
    auto issue = [&](int i) __attribute__((always_inline)) { issue_at(entry0(i), i % kSlots); };

    // Decode of four columns of a landed batch. The bitmap words come from
    // scalar loads of the bitmap array (the batch's DMA has just brought their
    // lines into L2) straight into scalar registers, where they serve as
    // MaskedPopcount masks and as EXEC masks of the value reads.
    const const_ptr<unsigned char> bitmap_s = (const_ptr<unsigned char>)bitmap;
    auto load_masks = [&](uint64_t (&m)[kQuad][WPC], uint32_t bo_v, int u0) __attribute__((always_inline)) {
  #pragma unroll
      for (int c = 0; c < kQuad; ++c) {
        const uint32_t bo = (uint32_t)__builtin_amdgcn_readlane((int)bo_v, u0 + c);
        const const_ptr<uint64_t> bp = (const_ptr<uint64_t>)(bitmap_s + bo);
  #pragma unroll
        for (int w = 0; w < WPC; ++w) m[c][w] = bp[w];
      }
    };
    auto decode_quad = [&](const unsigned char* slot, int e0, int u0, const uint64_t (&m)[kQuad][WPC], int half)
        __attribute__((always_inline)) {
      // 3. bitmap decode: a row's value sits at the MaskedPopcount of its word
      // below the lane plus the popcounts of the column's earlier words (every
      // lane reads; lanes whose bit is clear read a neighbour inside the slot
      // and are masked off below)
      uint32_t vb[kQuad][WPC];
  #pragma unroll
      for (int c = 0; c < kQuad; ++c) {
        // running LDS byte address of the word's first value (scalar): one
        // popcount and one shift-add per word
        uint32_t sb = lds_addr(slot + (u0 + c) * kSlotBytes);
  #pragma unroll
        for (int w = 0; w < WPC; ++w) {
          if constexpr (Q) {
            // a code is one byte: no shift in the address (an add instead:
            // the mbcnt cannot take both the mask and the base from scalar
            // registers); the signed code becomes an fp16 integer (exact for
            // |q| <= 127), and the rest of the decode is that of fp16 values
            const uint32_t a = sb + mbcnt64(m[c][w]);
            const int q = *(const __attribute__((address_space(3))) int8_t*)(uintptr_t)a;
            vb[c][w] = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)(int16_t)q);
            if (w + 1 < WPC) sb += (uint32_t)__builtin_popcountll(m[c][w]);
          } else {
            const uint32_t a = sb + 2u * mbcnt64(m[c][w]);
            vb[c][w] = *(const __attribute__((address_space(3))) uint16_t*)(uintptr_t)a;
            if (w + 1 < WPC) {
              const uint32_t pop = (uint32_t)__builtin_popcountll(m[c][w]);
              asm("s_lshl1_add_u32 %0, %1, %0" : "+s"(sb) : "s"(pop) : "scc");
            }
          }
        }
      }
      // 4. accumulate in fp32. One or two tokens: the words become EXEC around
      // single FMAs (v_fma_mix, fp16 operands; no branch, no select), NB per
      // word. From four tokens on the quad's four columns times four tokens
      // are a small dense contraction per 64-row word: the two columns of a
      // pair are selected into the halves of one register (zero where the bit
      // is clear: one SDWA select per column word), and one
      // v_mfma_f32_4x4x4_16b_f16 per word and four tokens adds the four
      // columns, in place of NB dot products (v_dot2) per column pair.
      if constexpr (MM) {
        // 4 (MFMA form). The batch's four columns, zero where the bit is
        // clear, into the wave's dense tile: row 64 w + lane, columns 4 h ..
        // 4 h + 3 for batch parity h (one 8-byte store per word); the
        // multiply runs once per two batches (below).
        unsigned char* mt = mt_s + wave * (64 * WPC * kMRowBytes);
  #pragma unroll
        for (int w = 0; w < WPC; ++w) {
          const uint32_t p01 = pair_under_words(vb[0][w], vb[1][w], m[0][w], m[1][w]);
          const uint32_t p23 = pair_under_words(vb[2][w], vb[3][w], m[2][w], m[3][w]);
          *reinterpret_cast<uint2*>(mt + (64 * w + lane) * kMRowBytes + 8 * half) = make_uint2(p01, p23);
        }
      } else if constexpr (NB == 2) {
  #pragma unroll
        for (int pr = 0; pr < 2; ++pr) {
          // the pair's dwords of tokens 0 and 1 (low half column 2pr)
          const uint2 xq = *reinterpret_cast<const uint2*>(&xs_s[((e0 + u0) / 2 + pr) * NB * 2]);
          masked_fma_column2<WPC, false>(acc, vb[2 * pr], xq.x, xq.y, m[2 * pr]);
          masked_fma_column2<WPC, true>(acc, vb[2 * pr + 1], xq.x, xq.y, m[2 * pr + 1]);
        }
      } else if constexpr (NB == 1) {
        const uint2 xq = *reinterpret_cast<const uint2*>(&xs_s[e0 + u0]);
  #pragma unroll
        for (int c = 0; c < kQuad; ++c) {
          const uint32_t xpair = c < 2 ? xq.x : xq.y;
          if (c & 1)
            masked_fma_column<WPC, true>(acc, vb[c], xpair, m[c]);
          else
            masked_fma_column<WPC, false>(acc, vb[c], xpair, m[c]);
        }
      } else {
        // four columns x four tokens per v_mfma_f32_4x4x4_16b_f16: B = the
        // quad's masked values of the lane's row (the two column pairs), A =
        // the quad's activations of token 4g + (lane & 3), so that lane r
        // gets rows r of tokens 4g .. 4g + 3 (D[4b + i][e] = sum_k A[4b + e][k]
        // B[4b + i][k])
        uint2 wv[WPC];
  #pragma unroll
        for (int w = 0; w < WPC; ++w)
          wv[w] = make_uint2(pair_under_words_mfma(vb[0][w], vb[1][w], m[0][w], m[1][w]),
                             pair_under_words_mfma(vb[2][w], vb[3][w], m[2][w], m[3][w]));
        const uint2* xq = reinterpret_cast<const uint2*>(&xs_s[((e0 + u0) / 4) * kXRow * 4]);
  #pragma unroll
        for (int g = 0; g < NB / 4; ++g) {
          const int t = 4 * g + (lane & 3);
          const half4_t xa = __builtin_bit_cast(half4_t, xq[t]);
  #pragma unroll
          for (int w = 0; w < WPC; ++w)
            acc4[w][g] = __builtin_amdgcn_mfma_f32_4x4x4f16(xa, __builtin_bit_cast(half4_t, wv[w]), acc4[w][g], 0, 0, 0);
        }
      }
    };
    static_assert(kQuad == 4, "decode works on quads of columns");

    // The ring: batches 0 .. kSlots-1 are requested up front; after batch i is
    // decoded its slot takes batch i + kSlots. Every batch is kDmaPerBatch
    // loads, so "batch i has landed" is "at most kDmaPerBatch x (batches
    // requested after i) loads outstanding". In the early-first-batch form
    // (small products, few waves per CU to hide latency with) and with more
    // than one token (measured: 0-2.5 % faster at 2-8 tokens, -2 to +1 % at
    // 16 and 32) the bitmap words
    // of batch i + 1 are requested as soon as batch i no longer needs their
    // registers, so that their round trip overlaps the wait for batch i + 1's
    // values; with many waves per CU, requesting them after that wait is
    // faster (measured: -2 to -3 % at 4096x4096 and 11008x4096 one way, +3 to
    // +6 % at 28672x8192 the other).
    static_assert(kBatch == kQuad, "a batch is one decode quad");
    for (int i = n_first; i < min(n_mine, kSlots); ++i) issue(i);
    uint64_t m[kQuad][WPC];
    auto masks_of = [&](int i) __attribute__((always_inline)) {
      // byte offsets of the batch's bitmaps: lane u < kBatch holds column u's
      const uint32_t bo_v = ent_bitmap(ent_s[entry0(i) + (lane & (kBatch - 1))].y);
      load_masks(m, bo_v, 0);
    };
    constexpr bool kAhead = EARLY || NB > 1;
    if (kAhead && n_mine > 0) masks_of(0);
    for (int i = 0; i < n_mine; ++i) {
      const int later = min(n_mine - 1 - i, kSlots - 1);
      if (later >= 3)
        wait_vmcnt<3 * kDmaPerBatch>();
      else if (later == 2)
        wait_vmcnt<2 * kDmaPerBatch>();
      else if (later == 1)
        wait_vmcnt<kDmaPerBatch>();
      else
        wait_vmcnt<0>();
      if (!kAhead) masks_of(i);
      decode_quad(my_ring + (i % kSlots) * kBatchBytes, entry0(i), 0, m, i & 1);
      if constexpr (MM) {
        // every second batch (and the last): the step's 8 columns (entries
        // e .. e + 7) times the 32 tokens: per 32-row block one
        // v_mfma_f32_32x32x8_f16, A = the tile's rows (lane l: row l mod 32,
        // columns 4 (l / 32) .. + 4), B = the columns' masked activations
        // (lane l: token l mod 32, the same 4 columns; 0 for tokens past NB)
        if ((i & 1) || i + 1 == n_mine) {
          unsigned char* mt = mt_s + wave * (64 * WPC * kMRowBytes);
          const int hl = lane >> 5;
          if (!(i & 1)) {
            // a single batch: the tile's second half is cleared (its columns
            // are the next wave's, and stale weights must not meet 0)
  #pragma unroll
            for (int w = 0; w < WPC; ++w) *reinterpret_cast<uint2*>(mt + (64 * w + lane) * kMRowBytes + 8) = make_uint2(0u, 0u);
          }
          const int e = entry0(i - (i & 1));
          const int t = lane & 31;
          uint2 bx = make_uint2(0u, 0u);
          if (t < NB && (hl == 0 || (i & 1))) {
            uint32_t h[4];
  #pragma unroll
            for (int j = 0; j < 4; ++j) {
              const uint32_t p = (uint32_t)(e + 4 * hl + j);
              h[j] = xs_s[p * NB + 8 * ((uint32_t)(t >> 3) ^ mm_swz(p)) + (t & 7)];
            }
            bx = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
          }
          const half4_t bop = __builtin_bit_cast(half4_t, bx);
          // the A operands are read together (one LDS round trip; the empty
          // asm keeps the compiler from interleaving each read with its
          // multiply)
          uint2 av[kMBlocks];
  #pragma unroll
          for (int blk = 0; blk < kMBlocks; ++blk)
            av[blk] = *reinterpret_cast<const uint2*>(mt + (32 * blk + t) * kMRowBytes + 8 * hl);
  #pragma unroll
          for (int blk = 0; blk < kMBlocks; ++blk) asm volatile("" ::"v"(av[blk]));
  #pragma unroll
          for (int blk = 0; blk < kMBlocks; ++blk)
            macc[blk] = __builtin_amdgcn_mfma_f32_32x32x8f16(__builtin_bit_cast(half4_t, av[blk]), bop, macc[blk], 0, 0, 0);
        }
      }
      if (i + kSlots < n_mine) {
        // the slot's LDS reads have completed (their results were consumed)
        issue(i + kSlots);
      }
      if (kAhead && i + 1 < n_mine) masks_of(i + 1);
    }

  }

  // ---- 5. reduce the 4 waves in LDS and publish this segment's partial
  // sums: device-coherent 8-byte stores, so that value and tag land together
  // and can be read from another XCD
  const_ptr<MatArgs> ka = &reload_args<LaunchArgs>()->m[mi];
  const int mpad = ka->n_stripes * ka->tile_m;
  const int n_seg = ka->segments;
  const int nb = batch;
  const int row = threadIdx.x;
  float* red = reinterpret_cast<float*>(ring);
  static_assert(!MM || kWaves * 32 * 32 * 4 <= S::kRingBytes, "the MFMA form's reduction reuses the ring");
  constexpr int kSlice = Smem<NB>::kSlice;
  unsigned long long* dst = ka->partials + (size_t)seg * nb * mpad + (size_t)r * ka->tile_m + row;
  const unsigned long long tag = (unsigned long long)phase << 32;
  if constexpr (MM) {
    // per 32-row block: each wave's 32 x 32 accumulators to LDS as
    // [wave][token][row], then thread (row, 4 tokens) adds the waves in
    // order 0..3 and publishes (consecutive threads, consecutive rows). A
    // stripe of one segment has nothing to gather: its sums are the rows'
    // results (0 + sum, the value the gather would produce) and go straight
    // to Y, and no partial, reducer or tag is involved.
    const int prow = threadIdx.x & 31;
    const int ptg = threadIdx.x >> 5;
    const bool direct = n_seg == 1;
    const int rows_d = ka->rows;
#pragma unroll
    for (int blk = 0; blk < kMBlocks; ++blk) {
      __syncthreads();
#pragma unroll
      for (int e = 0; e < 16; ++e)
        red[(wave * 32 + (lane & 31)) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)] = macc[blk][e];
      __syncthreads();
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const int b = 4 * ptg + bb;
        if (b < nb) {
          float sum = 0.0f;
#pragma unroll
          for (int wv = 0; wv < kWaves; ++wv) sum += red[(wv * 32 + b) * 32 + prow];
          const int m = r * ka->tile_m + 32 * blk + prow;
          if (!direct)
            __hip_atomic_store(dst - row + 32 * blk + prow + (size_t)b * mpad, tag | __float_as_uint(sum),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          else if (m < rows_d)
            ka->y[(size_t)b * rows_d + m] = __half_as_ushort(__float2half_rn(0.0f + sum));
        }
      }
    }
    if (direct) return;
  }
  // the vector-ALU forms: per token slice, the waves' accumulators to LDS,
  // then thread `row` adds them in wave order and publishes; a stripe of one
  // segment writes Y as the MFMA form does (the row scale applied as the
  // gather applies it)
  const bool direct_v = !MM && n_seg == 1;
  const int m_v = r * ka->tile_m + row;
  const bool live_v = row < 64 * WPC && m_v < ka->rows;
  const float scale_v = (Q && direct_v && live_v) ? ka->scales[m_v] : 1.0f;
#pragma unroll
  for (int b0 = 0; b0 < (MM ? 0 : NB); b0 += kSlice) {
    __syncthreads();
#pragma unroll
    for (int w = 0; w < WPC; ++w)
#pragma unroll
      for (int bb = 0; bb < kSlice; ++bb)
        red[(wave * kSlice + bb) * 256 + 64 * w + lane] = kM4 ? acc4[w][(b0 + bb) / 4][(b0 + bb) % 4] : acc[w][b0 + bb];
    __syncthreads();
#pragma unroll
    for (int bb = 0; bb < kSlice; ++bb) {
      if (row < 64 * WPC && b0 + bb < nb) {
        float s = 0.0f;
#pragma unroll
        for (int wv = 0; wv < kWaves; ++wv) s += red[(wv * kSlice + bb) * 256 + row];
        if (!direct_v) {
          __hip_atomic_store(dst + (size_t)(b0 + bb) * mpad, tag | __float_as_uint(s), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        } else if (live_v) {
          float t = 0.0f + s;
          if constexpr (Q) t *= scale_v;
          ka->y[(size_t)(b0 + bb) * ka->rows + m_v] = __half_as_ushort(__float2half_rn(t));
        }
      }
    }
  }
  if (direct_v) return;

  // ---- the stripe's last n_red segments gather: reducer j owns the 64-row
  // blocks w = j, j + n_red, ...; its four waves split the segments (wave g
  // takes segments g, g+4, ...), request all of a chunk of them at once,
  // request again those not yet tagged with this call's phase, and add them
  // in order; the four wave sums are added in wave order, so the result does
  // not depend on timing. The workgroups of lower segments of the stripe were
  // dispatched before these, so the wait ends; a bound on the rounds still
  // makes every wave exit (the rows then read NaN).
  // Reducers take units (64-row block w, token slice): a slice is every
  // token up to 8 tokens, and 8 tokens beyond; unit u = w + WPC x slice goes
  // to reducer u mod n_red. Splitting the tokens keeps several segments of
  // a slice in flight per round at large batches (one segment per round for
  // 16 or 32 tokens would cost a device-scope round trip per segment) and
  // spreads the gather over more workgroups; the sum per token is the same.
  constexpr bool kSliced = NB > 8;
  constexpr int kTok = kSliced ? 8 : NB;
  const int n_units = kSliced ? WPC * ((nb + kTok - 1) / kTok) : WPC;
  const int n_red = min(n_seg, n_units);
  const int jr = seg - (n_seg - n_red);
  if (jr < 0) return;
  // A round requests kJ of the wave's segments for every token of the slice
  // at once (about kGather partials in flight per lane: 16 where the
  // kernel's occupancy is bound by LDS and the registers are free, 12 at
  // one token, where they are not).
  constexpr int kGather = NB > 8 ? NB : NB >= 2 ? 16 : 12;
  constexpr int kJ = kGather / kTok >= 1 ? kGather / kTok : 1;
  constexpr int kMaxRounds = 1 << 22;
  const int rows = ka->rows;
  for (int u = jr; u < n_units; u += n_red) {
    const int w = kSliced ? u % WPC : u;
    const int b0 = kSliced ? (u / WPC) * kTok : 0;
    const int m = r * ka->tile_m + 64 * w + lane;
    const bool live = m < rows;
    const unsigned long long* src = ka->partials + (live ? m : 0);
    // Q form: the row's scale, requested ahead of the partials
    const float row_scale = Q ? (live ? ka->scales[m] : 0.0f) : 1.0f;
    float sums[kTok];
#pragma unroll
    for (int b = 0; b < kTok; ++b) sums[b] = 0.0f;
    if (live) {
      bool lost = false;
      auto part = [&](int sg, int b) {
        return __hip_atomic_load(src + ((size_t)sg * nb + b0 + b) * mpad, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
      };
      // this wave's segments: wave, wave + 4, ...
      for (int sg0 = wave; sg0 < n_seg; sg0 += kWaves * kJ) {
        unsigned long long v[kJ][kTok];
#pragma unroll
        for (int jj = 0; jj < kJ; ++jj)
#pragma unroll
          for (int b = 0; b < kTok; ++b)
            if (b0 + b < nb) v[jj][b] = part(min(sg0 + kWaves * jj, n_seg - 1), b);
        for (int round = 0;; ++round) {
          bool ready = true;
#pragma unroll
          for (int jj = 0; jj < kJ; ++jj)
#pragma unroll
            for (int b = 0; b < kTok; ++b)
              if (b0 + b < nb && sg0 + kWaves * jj < n_seg && (uint32_t)(v[jj][b] >> 32) != phase) {
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
          for (int b = 0; b < kTok; ++b)
            if (b0 + b < nb && sg0 + kWaves * jj < n_seg) sums[b] += __uint_as_float((uint32_t)v[jj][b]);
      }
      if (lost)
#pragma unroll
        for (int b = 0; b < kTok; ++b) sums[b] = __builtin_nanf("");
    }
#pragma unroll
    for (int b = 0; b < kTok; ++b) {
      if (b0 + b < nb) {  // uniform over the workgroup
        __syncthreads();
        red[wave * 64 + lane] = sums[b];
        __syncthreads();
        if (wave == 0 && live) {
          float t = ((red[lane] + red[64 + lane]) + red[128 + lane]) + red[192 + lane];
          if constexpr (Q) t *= row_scale;  // y = s * sum q x, rounded once to fp16
          ka->y[(size_t)(b0 + b) * rows + m] = __half_as_ushort(__float2half_rn(t));
        }
      }
    }
  }
  // Reducer 0 gathers row 0 of the stripe, a row that always exists (the
  // last reducer's rows can all lie past a ragged end, and it would then wait
  // for nothing), and its four waves together wait for every segment, so past
  // its barriers every workgroup of the stripe has published, and so has
  // read the phase; the next call starts after this kernel ends: advance the
  // tag (0 is skipped, the workspace's initial contents). The other reducers
  // keep their own copies of the phase. With the device-wide epoch the same
  // holds for every stripe once each stripe's first reducer has counted
  // itself: the last of them stores this call's tag as the epoch (the next
  // call tags with one more) and clears the count for the next call.
  if (jr == 0 && threadIdx.x == 0) {
    uint32_t* const done = ka->epoch_done;
    if (done == nullptr) {
      ka->phase[r] = phase + 1u == 0u ? 1u : phase + 1u;
    } else if (__hip_atomic_fetch_add(done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               (uint32_t)ka->n_stripes - 1u) {
      __hip_atomic_store(done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(ka->phase, phase, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// The kernels: the vector-ALU forms, and the matrix-core form, whose 32 x 32
// accumulator blocks live in AGPRs; two waves per SIMD are asked of it.
template <int NB, int WPC, bool EARLY, bool BMASK, bool Q, bool MP, int MWC>
__global__ __launch_bounds__(kThreads) void spmspv_kernel(LaunchArgs) {
  spmspv_body<NB, WPC, EARLY, BMASK, Q, false, MP, MWC>();
}
template <int NB, int WPC, bool BMASK, int MWC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void spmspv_mm_kernel(LaunchArgs) {
  spmspv_body<NB, WPC, false, BMASK, false, true, true, MWC>();
}

using spdp::fail;

int hip_fail(hipError_t e, const char* what) {
  return fail(SPDP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Split-K heuristic. Each wave tests and streams a K range of wave_cols
// columns (a multiple of 16); a product's grid is stripes x segments with
// segments = ceil(cols / (4 wave_cols)). Measured on the Llama shapes (sweeps
// of the segment count): 48 columns per wave; then the range widens in steps
// of 16 columns (to at most kMaxWaveCols) while there are more segments than
// one gather round reads at batch 1 (four waves x 12 partials in flight: a
// second round is a second device-scope round trip, about 1.5 us) or more
// than 1792 workgroups (the seven per CU that fit at once), and narrows
// while there are fewer than 512 (two per CU). This gives 4096x4096: 32
// segments, 5120x5120: 27, 4096x11008: 43, 5120x13824: 44, 11008x4096: 22,
// 13824x5120: 27, 28672x8192: 16. The split is a property of the product
// alone (it fixes the summation order), so a grouped launch adds up the
// products' workgroups: 40 segments would make a lone 5120x5120 product 6 %
// faster but three of them (q, k, v) in one launch 5 % slower.
// SPDP_SPLITK overrides the number of segments (for tuning).
constexpr int kWaveCols = 48;
constexpr int64_t kOneRoundSegments = 48;
constexpr int64_t kMinWorkgroups = 512;
constexpr int64_t kMaxWorkgroups = 1792;
// The 32x32 matrix-core form (a 32-row block x 32 tokens per instruction)
// runs only when SPDP_MFMA=1 asks for it, from 5 tokens on: the vector forms
// (one 4x4x4 product per 64-row word and four tokens from 3 tokens on) are
// as fast or faster at every measured size, at 32 tokens per product on one
// box, both with the passes below, on the Llama-70B layer 92.0 against
// 93.3 us (70/50) and 91.7 against 95.9 (50/0), the Llama-13B layer 50.4
// against 53.1, the Llama-7B MLP 51.6 against 55.6. A property of the batch
// only, so a product gives the same bits alone and grouped.
bool use_mfma(int batch) {
  if (batch < 5) return false;
  if (const char* env = std::getenv("SPDP_MFMA")) return std::atoi(env) != 0;
  return false;
}

// Passes per workgroup: more passes mean fewer segments, so fewer split-K
// partials (segments x batch x rows x 8 bytes, written and read back), and
// fewer, longer workgroups. The rule takes the largest P of 4, 2, 1 whose
// workgroups W_P (stripes x segments / P, rounded up) satisfy
// W_P x batch >= 2560 P: the partials' bytes grow with the batch, the cost of
// too few workgroups with P. Measured per product at 8 / 16 tokens with 1, 2
// or 4 passes everywhere: Llama-70B layer 46.7 / 43.1 / 50.2 and 58.4 / 51.6 /
// 58.0 us, Llama-13B 23.4 / 24.1 / 30.6 and 31.9 / 29.9 / 36.1, Llama-7B MLP
// (8 tokens) 24.9 / 25.7 / 37.3; at 32 tokens the rule (4 passes on the
// Llama-70B products but k and v, 2 on most others) is within 1-3 % of the
// best uniform count on each layer (the Llama-7B MLP at 4 passes everywhere:
// 46 % slower: 516 workgroups in the grouped gate/up launch against 512
// resident at two per CU). One or two tokens and the code forms walk one range. SPDP_PASSES
// overrides (for tuning). A property of the matrix and the batch, like the
// split, so a product gives the same bits alone and grouped.
int passes_for(int batch, bool codes, int64_t stripes, int64_t segs) {
  if (codes || batch < 3) return 1;
  if (const char* env = std::getenv("SPDP_PASSES")) {
    const long v = std::strtol(env, nullptr, 10);
    if (v >= 1 && v <= 64) return (int)v;
  }
  for (int p = 4; p > 1; p /= 2)
    if (stripes * ((segs + p - 1) / p) * batch >= int64_t(2560) * p) return p;
  return 1;
}

void choose_split(const spdp_matrix* m, int batch, int* segments, int* wave_cols, int* passes) {
  const int64_t cols = std::max<int64_t>(1, m->cols);
  const int64_t stripes = std::max<int64_t>(1, m->n_stripes);
  auto segs = [&](int64_t wc) { return (cols + kWaves * wc - 1) / (kWaves * wc); };
  int64_t wc = kWaveCols;
  const bool codes = m->value_bits < 16;
  if (const char* env = std::getenv("SPDP_SPLITK")) {
    const long v = std::strtol(env, nullptr, 10);
    if (v >= 1) {
      wc = std::min<int64_t>(kMaxWaveCols, ((cols + v * kWaves - 1) / (v * kWaves) + 15) / 16 * 16);
      *wave_cols = (int)wc;
      *passes = passes_for(batch, codes, stripes, segs(wc));
      *segments = (int)((segs(wc) + *passes - 1) / *passes);
      return;
    }
  }
  while ((stripes * segs(wc) > kMaxWorkgroups || segs(wc) > kOneRoundSegments) && wc < kMaxWaveCols) wc += 16;
  while (stripes * segs(wc) < kMinWorkgroups && wc > 16 && segs(wc - 16) <= kOneRoundSegments) wc -= 16;
  *wave_cols = (int)wc;
  *passes = passes_for(batch, codes, stripes, segs(wc));
  *segments = (int)((segs(wc) + *passes - 1) / *passes);
}

// The workspace holds {fp32, phase} pairs for all segments; it starts zeroed
// and phases are never 0, so nothing in it matches a call before that call
// has written it. Growing it never waits for the device and never frees: the
// old workspace may still be read by work in flight or named by a captured
// graph, so it is kept until spdp_free. On the call path (stream given) the
// new one is cleared on the call's stream, ahead of the kernel; inside a
// stream capture no allocation is made at all (the call is refused: size
// the workspace with spdp_reserve before capturing).
int ensure_workspace(spdp_matrix* m, int batch, int segments, bool on_call, hipStream_t stream) {
  const size_t need = (size_t)segments * batch * m->n_stripes * m->tile_m;
  if (need <= m->partial_floats) return SPDP_OK;
  if (on_call) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(stream, &cs);
    if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
    if (cs != hipStreamCaptureStatusNone)
      return fail(SPDP_ERR_INVALID_ARG,
                  "the split-K workspace is too small for this batch and the stream is capturing; "
                  "call spdp_reserve(h, batch) before the capture");
  }
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, need * sizeof(unsigned long long));
  if (e != hipSuccess)
    return e == hipErrorOutOfMemory ? fail(SPDP_ERR_OOM, "hipMalloc of the split-K workspace failed")
                                    : hip_fail(e, "hipMalloc");
  e = on_call ? hipMemsetAsync(p, 0, need * sizeof(unsigned long long), stream)
              : hipMemset(p, 0, need * sizeof(unsigned long long));
  if (e != hipSuccess) {
    (void)hipFree(p);
    return hip_fail(e, "hipMemset");
  }
  if (m->d_partials) m->retired.push_back(m->d_partials);
  m->d_partials = static_cast<unsigned long long*>(p);
  m->partial_floats = need;
  return SPDP_OK;
}

void release_device(spdp_matrix* m) {
  if (m->device < 0) return;
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(m->device);
  (void)hipDeviceSynchronize();
  void* ptrs[] = {m->d_tile_offset, m->d_col_info, m->d_bitmap, m->d_values, m->d_scales, m->d_partials, m->d_phase,
                  m->d_spmm_part};
  for (void* p : ptrs)
    if (p) (void)hipFree(p);
  for (void* p : m->retired) (void)hipFree(p);
  m->retired.clear();
  m->d_tile_offset = m->d_col_info = m->d_bitmap = m->d_values = m->d_scales = nullptr;
  m->d_partials = nullptr;
  m->d_phase = nullptr;
  m->partial_floats = 0;
  m->d_spmm_part = nullptr;
  m->spmm_part_bytes = 0;
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

template <int NB, int WPC, bool Q, int MWC>
hipError_t launch_cols(const LaunchArgs& args, bool early, bool bmask, bool mm, bool multi, dim3 grid,
                       hipStream_t stream) {
  // the one-token kernel has the early-first-batch form (no product with
  // more tokens asks for it); the kernels for more tokens have the shared
  // batch mask form (at one token the two masks are the same rule, and the
  // host sends such calls to the per-token kernel); from 8 tokens on, fp16
  // values accumulate in 32x32 blocks when mm is set; from 4, the kernels
  // for fp16 values have a several-range form (multi: some product of the
  // launch walks more than one K range; one range in it gives the bits of
  // the one-range kernel)
  if constexpr (NB == 1) {
    if (early) {
      hipLaunchKernelGGL((spmspv_kernel<NB, WPC, true, false, Q, false, MWC>), grid, dim3(kThreads), 0, stream, args);
      return hipGetLastError();
    }
  } else {
    if constexpr (NB >= 8 && !Q) {
      if (mm) {
        if (bmask)
          hipLaunchKernelGGL((spmspv_mm_kernel<NB, WPC, true, MWC>), grid, dim3(kThreads), 0, stream, args);
        else
          hipLaunchKernelGGL((spmspv_mm_kernel<NB, WPC, false, MWC>), grid, dim3(kThreads), 0, stream, args);
        return hipGetLastError();
      }
    }
    if constexpr (NB >= 4 && !Q) {
      if (multi) {
        if (bmask)
          hipLaunchKernelGGL((spmspv_kernel<NB, WPC, false, true, Q, true, MWC>), grid, dim3(kThreads), 0, stream,
                             args);
        else
          hipLaunchKernelGGL((spmspv_kernel<NB, WPC, false, false, Q, true, MWC>), grid, dim3(kThreads), 0, stream,
                             args);
        return hipGetLastError();
      }
    }
    if (bmask) {
      hipLaunchKernelGGL((spmspv_kernel<NB, WPC, false, true, Q, false, MWC>), grid, dim3(kThreads), 0, stream, args);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((spmspv_kernel<NB, WPC, false, false, Q, false, MWC>), grid, dim3(kThreads), 0, stream, args);
  return hipGetLastError();
}

// wide: some product of the launch tests more than 64 columns per range
template <int NB, int WPC, bool Q>
hipError_t launch_form(const LaunchArgs& args, bool early, bool bmask, bool mm, bool multi, bool wide, dim3 grid,
                       hipStream_t stream) {
  if (NB == 1 || wide) return launch_cols<NB, WPC, Q, kMaxWaveCols>(args, early, bmask, mm, multi, grid, stream);
  if constexpr (NB > 1) return launch_cols<NB, WPC, Q, kNarrowWaveCols>(args, early, bmask, mm, multi, grid, stream);
  return hipErrorInvalidValue;
}

template <int NB, int WPC>
hipError_t launch_one(const LaunchArgs& args, bool early, bool bmask, bool mm, bool multi, bool wide, bool q,
                      dim3 grid, hipStream_t stream) {
  return q ? launch_form<NB, WPC, true>(args, early, bmask, mm, multi, wide, grid, stream)
           : launch_form<NB, WPC, false>(args, early, bmask, mm, multi, wide, grid, stream);
}

template <int NB>
hipError_t launch(const LaunchArgs& args, int wpc, bool early, bool bmask, bool mm, bool multi, bool wide, bool q,
                  dim3 grid, hipStream_t stream) {
  switch (wpc) {
    case 1: return launch_one<NB, 1>(args, early, bmask, mm, multi, wide, q, grid, stream);
    case 2: return launch_one<NB, 2>(args, early, bmask, mm, multi, wide, q, grid, stream);
    case 3: return launch_one<NB, 3>(args, early, bmask, mm, multi, wide, q, grid, stream);
    default: return launch_one<NB, 4>(args, early, bmask, mm, multi, wide, q, grid, stream);
  }
}


// Early first batches (each wave requests its own first four active columns
// before the workgroup builds its list) pay where a product is latency-bound:
// measured -6 % on a lone 4096x4096 product (512 workgroups), -2 % at
// 11008x4096 (946); with five or more workgroups per CU, or with more than
// one token, the latency is hidden anyway and the extra prologue work costs
// 1-3 %. Decided per product (its own workgroups), so that a product gives
// the same bits alone and in a group. SPDP_EARLY_FIRST=0 or 1 overrides (for
// tuning).
constexpr int64_t kEarlyFirstMaxWorkgroups = 1024;
int early_first(int batch, int64_t workgroups) {
  if (batch != 1) return 0;  // the form exists for one token only
  if (const char* env = std::getenv("SPDP_EARLY_FIRST")) return std::atoi(env) != 0 ? 1 : 0;
  return workgroups <= kEarlyFirstMaxWorkgroups ? 1 : 0;
}

// A split-K workspace that is not the handle's own: the library's static
// one (partials and the device-wide epoch with its stripe count).
struct SharedWorkspace {
  unsigned long long* partials;
  size_t capacity;  // pairs
  uint32_t* epoch;
  uint32_t* epoch_done;
};

// Validates one product of a call and fills its kernel arguments: with the
// handle's workspace (sized for the batch if needed), or with `shared`.
int prepare(spdp_handle_t h, const uint16_t* X, int32_t batch, float threshold, int32_t mask, uint16_t* Y, int dev,
            hipStream_t stream, const SharedWorkspace* shared, MatArgs* out, int64_t* n_wg) {
  if (!h) return fail(SPDP_ERR_INVALID_ARG, "handle is NULL");
  if (h->device < 0) return fail(SPDP_ERR_INVALID_ARG, "handle has no device copy");
  if (!X || !Y) return fail(SPDP_ERR_INVALID_ARG, "X or Y is NULL");
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
  if (dev != h->device) return fail(SPDP_ERR_INVALID_ARG, "current device differs from the handle's");

  int segments = 1, wave_cols = 16, passes = 1;
  choose_split(h, batch, &segments, &wave_cols, &passes);
  if (shared) {
    const size_t need = (size_t)segments * batch * h->n_stripes * h->tile_m;
    if (need > shared->capacity)
      return fail(SPDP_ERR_UNSUPPORTED, "the product needs " + std::to_string(need * 8) +
                                            " bytes of split-K partials; the static workspace holds " +
                                            std::to_string(shared->capacity * 8));
  } else {
    st = ensure_workspace(h, batch, segments, true, stream);
    if (st != SPDP_OK) return st;
  }

  MatArgs& a = *out;
  a.tile_offset = static_cast<const uint32_t*>(h->d_tile_offset);
  a.col_info = static_cast<const uint32_t*>(h->d_col_info);
  a.bitmap = static_cast<const uint64_t*>(h->d_bitmap);
  a.values = static_cast<const uint16_t*>(h->d_values);
  a.scales = static_cast<const float*>(h->d_scales);
  a.x = X;
  a.y = Y;
  a.partials = shared ? shared->partials : h->d_partials;
  a.phase = shared ? shared->epoch : h->d_phase;
  a.epoch_done = shared ? shared->epoch_done : nullptr;
  a.phase_step = shared ? 0 : 1;
  a.rows = (int)h->rows;
  a.cols = (int)h->cols;
  a.tile_m = h->tile_m;
  a.zero_col = (uint32_t)(h->n_gtiles * h->tile_k);
  a.tk_log2 = __builtin_ctz((unsigned)h->tile_k);
  a.n_colblocks = (int)h->n_colblocks;
  a.n_stripes = (int)h->n_stripes;
  a.code = code;
  a.wave_cols = wave_cols;
  a.segments = segments;
  a.passes = passes;
  *n_wg = (int64_t)segments * h->n_stripes;
  a.n_wg = (int)*n_wg;
  a.early_first = early_first(batch, *n_wg);
  a.batch_thr = mask == SPDP_MASK_BATCH ? (float)((double)threshold * (double)batch) : 0.0f;
  return SPDP_OK;
}

bool overlap(const void* p, size_t pn, const void* q, size_t qn) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(p), b0 = reinterpret_cast<uintptr_t>(q);
  return a0 < b0 + qn && b0 < a0 + pn;
}

// Uploads the host arrays of a freshly encoded matrix to the current device
// and sizes its workspace for one token; on failure frees what it made and
// the matrix itself.
int finish_device(spdp_matrix* m, spdp_handle_t* out) {
  // the kernel packs a GTile column index (the all-zero padding column
  // included) into 26 bits and addresses values and bitmaps with 32-bit
  // byte offsets
  if (m->n_gtiles * m->tile_k + 1 >= (int64_t(1) << 26)) {
    delete m;
    return fail(SPDP_ERR_UNSUPPORTED, "more than 2^26 - 2 GTile columns (row stripes x padded columns)");
  }
  const uint64_t value_bytes = m->value_bits < 16 ? (uint64_t)m->codes.size() : (uint64_t)m->values.size() * 2;
  if (value_bytes + kTailBytes >= (uint64_t(1) << 32)) {
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
  int st = upload(m->tile_offset, &m->d_tile_offset);
  if (st == SPDP_OK) st = upload(m->col_info, &m->d_col_info);
  if (st == SPDP_OK) st = upload(m->bitmap, &m->d_bitmap);
  if (st == SPDP_OK) st = m->value_bits < 16 ? upload(m->codes, &m->d_values) : upload(m->values, &m->d_values);
  if (st == SPDP_OK && m->value_bits < 16) st = upload(m->scales, &m->d_scales);
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
    int segments = 1, wave_cols = 16, passes = 1;
    choose_split(m, 1, &segments, &wave_cols, &passes);
    st = ensure_workspace(m, 1, segments, false, nullptr);
  }
  if (st != SPDP_OK) {
    release_device(m);
    delete m;
    return st;
  }
  *out = m;
  return SPDP_OK;
}

// The launch behind every spMspV entry point: validates all products, then
// enqueues one kernel; `shared` selects the static workspace (one product).
int launch_products(const spdp_handle_t* handles, int32_t count, const uint16_t* const* X, int32_t batch,
                    const float* thresholds, int32_t mask, uint16_t* const* Y, void* stream,
                    const SharedWorkspace* shared) {
  if (!handles || !X || !Y || !thresholds) return fail(SPDP_ERR_INVALID_ARG, "an argument array is NULL");
  if (mask != SPDP_MASK_TOKEN && mask != SPDP_MASK_BATCH)
    return fail(SPDP_ERR_INVALID_ARG, "mask must be SPDP_MASK_TOKEN or SPDP_MASK_BATCH");
  if (count < 1 || count > kMaxGroup) return fail(SPDP_ERR_INVALID_ARG, "count must lie in [1, 8]");
  if (batch < 1 || batch > kMaxBatch) return fail(SPDP_ERR_INVALID_ARG, "batch must lie in [1, 32]");
  for (int i = 0; i < count; ++i) {
    if (!handles[i]) return fail(SPDP_ERR_INVALID_ARG, "handle is NULL");
    if (handles[i]->device < 0) return fail(SPDP_ERR_INVALID_ARG, "handle has no device copy");
  }
  for (int i = 0; i < count; ++i) {
    for (int j = 0; j < i; ++j) {
      if (handles[i] == handles[j])
        return fail(SPDP_ERR_INVALID_ARG, "a handle appears twice in one call (its workspace is shared)");
      {
        const size_t xi = (size_t)batch * handles[i]->cols * 2, yi = (size_t)batch * handles[i]->rows * 2;
        const size_t xj = (size_t)batch * handles[j]->cols * 2, yj = (size_t)batch * handles[j]->rows * 2;
        if (overlap(Y[i], yi, Y[j], yj) || overlap(Y[i], yi, X[j], xj) || overlap(Y[j], yj, X[i], xi))
          return fail(SPDP_ERR_INVALID_ARG, "an output overlaps another product's input or output");
      }
    }
  }
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  LaunchArgs la;
  std::memset(&la, 0, sizeof(la));
  la.batch = batch;
  int64_t widest = 0;
  bool early = false, multi = false, wide = false;
  const bool bmask = mask == SPDP_MASK_BATCH && batch > 1;
  for (int i = 0; i < count; ++i) {
    int64_t n_wg = 0;
    const int st = prepare(handles[i], X[i], batch, thresholds[i], mask, Y[i], dev, static_cast<hipStream_t>(stream),
                           shared, &la.m[i], &n_wg);
    if (st != SPDP_OK) return st;
    if (handles[i]->tile_m != handles[0]->tile_m)
      return fail(SPDP_ERR_INVALID_ARG, "the matrices of one call must share tile_m");
    if ((handles[i]->value_bits < 16) != (handles[0]->value_bits < 16))
      return fail(SPDP_ERR_INVALID_ARG, "the matrices of one call must all hold fp16 values or all codes");
    if (n_wg >= (int64_t(1) << 31)) return fail(SPDP_ERR_UNSUPPORTED, "more than 2^31 - 1 workgroups");
    widest = std::max(widest, n_wg);
    early = early || la.m[i].early_first;
    multi = multi || la.m[i].passes > 1;
    wide = wide || la.m[i].wave_cols > kNarrowWaveCols;
  }

  const int wpc = handles[0]->tile_m / 64;
  const dim3 grid((unsigned)widest, (unsigned)count);
  const bool q = handles[0]->value_bits < 16;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool mm = use_mfma(batch);
  if (batch <= 1)
    e = launch<1>(la, wpc, early, bmask, mm, multi, wide, q, grid, s);
  else if (batch <= 2)
    e = launch<2>(la, wpc, early, bmask, mm, multi, wide, q, grid, s);
  else if (batch <= 4)
    e = launch<4>(la, wpc, early, bmask, mm, multi, wide, q, grid, s);
  else if (batch <= 8)
    e = launch<8>(la, wpc, early, bmask, mm, multi, wide, q, grid, s);
  else if (batch <= 16)
    e = launch<16>(la, wpc, early, bmask, mm, multi, wide, q, grid, s);
  else
    e = launch<32>(la, wpc, early, bmask, mm, multi, wide, q, grid, s);
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return SPDP_OK;
}

// The static split-K workspace of spdp_spmspv_noalloc, for callers that
// cannot allocate device memory. Bytes [0, 256) hold the device-wide epoch
// (byte 0) and the count of stripes done with it (byte 128); the partials
// follow. Static storage starts zeroed, so no partial carries a live tag
// before a call writes it. Host code never uses the name `scratch` as an
// address (on the host it stands for the symbol): the device address comes
// from hipGetSymbolAddress, once per device.
constexpr size_t kScratchHeaderBytes = 256;
constexpr size_t kScratchPartialBytes = SPDP_NOALLOC_PARTIAL_BYTES;
static __device__ __align__(256) unsigned long long scratch[(kScratchHeaderBytes + kScratchPartialBytes) / 8];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch` (dev is current).
int scratch_on(int dev, SharedWorkspace* ws) {
  if (dev < 0 || dev >= kMaxDevices) return fail(SPDP_ERR_UNSUPPORTED, "device ordinal beyond 63");
  void* p = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
      hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
      if (!p) return fail(SPDP_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
      g_scratch_ptr[dev] = p;
    }
    p = g_scratch_ptr[dev];
  }
  char* base = static_cast<char*>(p);
  ws->epoch = reinterpret_cast<uint32_t*>(base);
  ws->epoch_done = reinterpret_cast<uint32_t*>(base + 128);
  ws->partials = reinterpret_cast<unsigned long long*>(base + kScratchHeaderBytes);
  ws->capacity = kScratchPartialBytes / sizeof(unsigned long long);
  return SPDP_OK;
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
  const int st = spdp::encode_host_arrays(W, rows, cols, tile_m, tile_k, m);
  if (st != SPDP_OK) {
    delete m;
    return st;
  }
  return finish_device(m, out);
}

int spdp_encode_rtn(const uint16_t* W, int64_t rows, int64_t cols, int32_t tile_m,
                    int32_t tile_k, int32_t bits, spdp_handle_t* out) {
  spdp::clear_error();
  if (!out) return fail(SPDP_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  spdp_matrix* m = new (std::nothrow) spdp_matrix();
  if (!m) return fail(SPDP_ERR_OOM, "host allocation failed");
  const int st = spdp::encode_host_arrays_rtn(W, rows, cols, tile_m, tile_k, bits, m);
  if (st != SPDP_OK) {
    delete m;
    return st;
  }
  return finish_device(m, out);
}

int spdp_reserve(spdp_handle_t h, int32_t max_batch) {
  spdp::clear_error();
  if (!h) return fail(SPDP_ERR_INVALID_ARG, "handle is NULL");
  if (h->device < 0) return fail(SPDP_ERR_INVALID_ARG, "handle has no device copy");
  if (max_batch < 1 || max_batch > kMaxBatch)
    return fail(SPDP_ERR_INVALID_ARG, "max_batch must lie in [1, 32]");
  // every batch up to max_batch: the split (and so the workspace) depends on it
  int64_t need = 0;  // segments x batch
  for (int b = 1; b <= max_batch; ++b) {
    int segments = 1, wave_cols = 16, passes = 1;
    choose_split(h, b, &segments, &wave_cols, &passes);
    need = std::max<int64_t>(need, (int64_t)segments * b);
  }
  return ensure_workspace(h, (int)need, 1, false, nullptr);
}

int spdp_split_plan(spdp_handle_t h, int32_t batch, int32_t* segments, int32_t* wave_cols, int32_t* passes) {
  spdp::clear_error();
  if (!h || !segments || !wave_cols || !passes) return fail(SPDP_ERR_INVALID_ARG, "handle or an output is NULL");
  if (batch < 1 || batch > kMaxBatch) return fail(SPDP_ERR_INVALID_ARG, "batch must lie in [1, 32]");
  int sg = 1, wc = 16, ps = 1;
  choose_split(h, batch, &sg, &wc, &ps);
  *segments = sg;
  *wave_cols = wc;
  *passes = ps;
  return SPDP_OK;
}

int spdp_spmspv_many_mask(const spdp_handle_t* handles, int32_t count, const uint16_t* const* X,
                          int32_t batch, const float* thresholds, int32_t mask, uint16_t* const* Y,
                          void* stream) {
  spdp::clear_error();
  return launch_products(handles, count, X, batch, thresholds, mask, Y, stream, nullptr);
}

int spdp_spmspv_many(const spdp_handle_t* handles, int32_t count, const uint16_t* const* X,
                     int32_t batch, const float* thresholds, uint16_t* const* Y, void* stream) {
  return spdp_spmspv_many_mask(handles, count, X, batch, thresholds, SPDP_MASK_TOKEN, Y, stream);
}

int spdp_spmspv(spdp_handle_t h, const uint16_t* X, int32_t batch, float threshold,
                uint16_t* Y, void* stream) {
  spdp::clear_error();
  return launch_products(&h, 1, &X, batch, &threshold, SPDP_MASK_TOKEN, &Y, stream, nullptr);
}

int spdp_spmspv_noalloc(spdp_handle_t h, const uint16_t* X, int32_t batch, float threshold,
                        uint16_t* Y, void* stream) {
  spdp::clear_error();
  if (!h) return fail(SPDP_ERR_INVALID_ARG, "handle is NULL");
  if (h->device < 0) return fail(SPDP_ERR_INVALID_ARG, "handle has no device copy");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != h->device) return fail(SPDP_ERR_INVALID_ARG, "current device differs from the handle's");
  SharedWorkspace ws;
  const int st = scratch_on(dev, &ws);
  if (st != SPDP_OK) return st;
  return launch_products(&h, 1, &X, batch, &threshold, SPDP_MASK_TOKEN, &Y, stream, &ws);
}

void spdp_free(spdp_handle_t h) {
  if (!h) return;
  release_device(h);
  delete h;
}

}  // extern "C"
