// Device side of libspdp for gfx950 (MI355X): the fused decode-time spMspV
// kernel over Tiled-CBC weights (Sec. 4.2) and the C-ABI entry points that
// own device memory.
//
// One launch per call does the whole path:
//   1. activity: each wave reads its slice of the activations and takes the
//      strict magnitude test |x| > t as an integer compare on fp16 bits; a
//      64-lane ballot turns the per-token results into a 64-column mask
//      (union over the batch) held in scalar registers (Sec. 4.2, XTile
//      loading and the activation-aware selection of GTile loading);
//   2. metadata then data (Sec. 4.2.2, "metadata first, data second"): the
//      scalar unit walks the set bits of the mask, loads each active column's
//      ColInfo and TileOffset entry with scalar loads, and the wave streams the
//      column's padded values with 16-byte vector loads into LDS, two columns
//      per load instruction (lanes 0-31 and 32-63);
//   3. bitmap decode (HAD-SMBD, Sec. 4.2.1): lane i owns row 64w+i of bitmap
//      word w; its value sits at the masked popcount of the word below bit i
//      (v_mbcnt_lo/hi, the MaskedPopcount of the paper) plus the popcount of
//      the earlier words, and the word itself is the execution mask, so rows
//      without a nonzero issue no LDS read and no FMA;
//   4. accumulate in fp32 on the vector ALUs with fp16 operands (v_fma_mix),
//      no matrix cores (Sec. 3.3 challenge 2, Sec. 4.2 step 5);
//   5. split-K (Sec. 4.2.3): the workgroups of a row stripe cover disjoint K
//      segments; each reduces its 4 waves in LDS and writes fp32 partial sums
//      to a workspace, and the last workgroup to arrive for the stripe adds
//      the partials in segment order and writes fp16 Y (round to nearest
//      even), then re-arms the stripe's counter for the next call.

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
constexpr int kLoadsPerBatch = kBatch / 2 + 1;  // 16-byte-per-lane loads issued per stage
constexpr int kMaxBatch = 32;

struct KernelArgs {
  const uint32_t* tile_offset;
  const uint32_t* col_info;
  const uint64_t* bitmap;
  const uint16_t* values;
  const uint16_t* x;
  uint16_t* y;
  float* partials;     // [segments][batch][n_stripes * tile_m]
  uint32_t* counters;  // [n_stripes], zero between calls
  int rows, cols;
  int tile_m, tk_log2, n_colblocks, n_stripes;
  int batch;
  int code;       // threshold code: active iff code < (x & 0x7fff) <= 0x7c00
  int wave_cols;  // columns per wave (multiple of 16, <= kMaxWaveCols)
  int segments;   // workgroups per row stripe
  uint32_t zero_col;  // column index whose bitmap lies in the zeroed tail padding
};

// LDS use. The two pipeline buffers are separate __shared__ arrays so that
// the compiler can tell reads of one from LDS-DMA writes into the other (it
// then waits only for the DMA a read depends on).
constexpr int kValBufBytes = kWaves * kBatch * kSlotBytes;  // one stage, all waves
constexpr int kBmBufBytes = kWaves * kBatch * 32;          // one stage, all waves

template <int NB>
struct Smem {
  static constexpr int kSlice = NB < 4 ? NB : 4;  // tokens per cross-wave reduction pass
  static constexpr int kRed = kWaves * kSlice * 256 * 4;
  static_assert(kRed <= kValBufBytes, "reduction reuses the first value buffer");
};

// s_waitcnt immediate for gfx9: wait until at most n vector-memory operations
// are outstanding, leaving the LDS/scalar and export counters unconstrained.
constexpr int vmcnt_imm(int n) { return (n & 0xF) | (((n >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8); }

__device__ __forceinline__ uint32_t mbcnt64(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return __half2float(__ushort_as_half((unsigned short)h));
}

// 16 bytes per lane from global memory straight into LDS: lane i's bytes land
// at lds_base + 16 * i (gfx950 LDS DMA).
__device__ __forceinline__ void lds_dma16(const void* src, void* lds_base) {
  __builtin_amdgcn_global_load_lds(src, reinterpret_cast<__attribute__((address_space(3))) void*>(
                                            reinterpret_cast<uintptr_t>(lds_base)),
                                   16, 0, 0);
}

// Read-only arrays reached through the constant address space: uniform
// (per-column) reads of them compile to scalar loads.
template <class T>
using const_ptr = const __attribute__((address_space(4))) T*;

template <class T>
__device__ __forceinline__ const_ptr<T> as_const(const T* p) {
  return reinterpret_cast<const_ptr<T>>(reinterpret_cast<uintptr_t>(p));
}

// Wave-uniform 64-bit value from two VGPR halves (readfirstlane yields int:
// go through uint32_t so that bit 31 of the low half is not sign-extended).
__device__ __forceinline__ uint64_t uniform64(uint32_t lo, uint32_t hi) {
  return (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane(lo) |
         ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane(hi) << 32);
}

// NB: tokens per call rounded up to a power of two; WPC: bitmap words per
// column (tile_m / 64).
template <int NB, int WPC>
__global__ __launch_bounds__(kThreads) void spmspv_kernel(KernelArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char val0[kValBufBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char val1[kValBufBytes];
  __shared__ __attribute__((aligned(256))) unsigned char bm0[kBmBufBytes];
  __shared__ __attribute__((aligned(256))) unsigned char bm1[kBmBufBytes];
  // one entry per active column, in activity order: {value base, column
  // index into ColInfo/bitmap, 16-byte chunks of values, unused}
  __shared__ uint4 ent_s[kWaves][kMaxWaveCols];
  __shared__ uint16_t xs_s[kWaves][kMaxWaveCols * NB];
  __shared__ __attribute__((aligned(16))) uint32_t col_s[kWaves][kMaxWaveCols];
  __shared__ int s_last;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int seg = blockIdx.x;
  const int r = blockIdx.y;
  const int tk_mask = (1 << a.tk_log2) - 1;
  const int g_row = r * a.n_colblocks;

  uint4* ent_l = ent_s[wave];
  uint16_t* xs_l = xs_s[wave];
  uint32_t* col_l = col_s[wave];
  unsigned char* my_val0 = val0 + wave * (kBatch * kSlotBytes);
  unsigned char* my_val1 = val1 + wave * (kBatch * kSlotBytes);
  unsigned char* my_bm0 = bm0 + wave * (kBatch * 32);
  unsigned char* my_bm1 = bm1 + wave * (kBatch * 32);

  float acc[WPC][NB];
#pragma unroll
  for (int w = 0; w < WPC; ++w)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[w][b] = 0.0f;

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
      ent_l[pos] = make_uint4(to[c] + (ci[c] >> 16), colx[c], ((ci[c] & 0xFFFFu) + 7u) >> 3, 0u);
      col_l[pos] = colx[c];
#pragma unroll
      for (int b = 0; b < NB; ++b) xs_l[pos * NB + b] = on[b] ? (uint16_t)xb[c][b] : (uint16_t)0;
    }
    n_act += __builtin_popcountll(act);
  }
  // Pad the last batch with entries that read an all-zero bitmap (in the
  // bitmap array's zeroed tail) and no values: they decode to nothing.
  if (lane < ((kBatch - (n_act & (kBatch - 1))) & (kBatch - 1)))
  {
    ent_l[n_act + lane] = make_uint4(0u, a.zero_col, 0u, 0u);
    col_l[n_act + lane] = a.zero_col;
  }

  // ---- 2. pipeline over batches of kBatch active columns: while batch i is
  // decoded, batch i+1's values and bitmaps are already streaming into LDS.
  const int n_batches = (n_act + kBatch - 1) / kBatch;
  const int hsel = lane >> 5;
  const int q = lane & 31;
  const unsigned char* bitmap_bytes = reinterpret_cast<const unsigned char*>(a.bitmap);

  auto issue = [&](int i, unsigned char* val_buf, unsigned char* bm_buf) {
    uint4 e[kBatch / 2];
#pragma unroll
    for (int pr = 0; pr < kBatch / 2; ++pr) e[pr] = ent_l[i * kBatch + 2 * pr + hsel];
    const uint4 eb = ent_l[i * kBatch + ((lane >> 1) & (kBatch - 1))];
    // values: lanes 0-31 fetch column 2pr, lanes 32-63 column 2pr+1, 16 B per
    // lane; lanes past the column's end re-read its first chunk (same cache
    // line) and what they leave in the slot is never read
#pragma unroll
    for (int pr = 0; pr < kBatch / 2; ++pr) {
      const int chunk = q < (int)e[pr].z ? q : 0;
      lds_dma16(a.values + (size_t)e[pr].x + 8 * chunk, val_buf + 2 * pr * kSlotBytes);
    }
    // bitmaps: lanes 2u and 2u+1 fetch the first and second 16 B of column u
    // (columns with fewer than 4 words read into the next column or the
    // arrays' tail padding; those words are never used)
    if (lane < 2 * kBatch) lds_dma16(bitmap_bytes + (size_t)eb.y * WPC * 8 + 16 * (lane & 1), bm_buf);
  };

  // The decode reads each quad's column indices from LDS, moves them to
  // scalar registers and loads the columns' bitmap words with scalar loads:
  // the words then serve directly as MaskedPopcount masks and EXEC masks.
  // (The LDS-DMA of the bitmaps above only pulls their lines into L2 ahead of
  // these loads.)
  const_ptr<uint64_t> bitmap_c = as_const(a.bitmap);

  auto decode = [&](int i, const unsigned char* val_buf) {
    const int n_here = min(kBatch, n_act - i * kBatch);
    for (int u0 = 0; u0 < n_here; u0 += kQuad) {
      const uint4 cq = *reinterpret_cast<const uint4*>(&col_l[i * kBatch + u0]);
      const uint32_t cols[kQuad] = {(uint32_t)__builtin_amdgcn_readfirstlane(cq.x),
                                    (uint32_t)__builtin_amdgcn_readfirstlane(cq.y),
                                    (uint32_t)__builtin_amdgcn_readfirstlane(cq.z),
                                    (uint32_t)__builtin_amdgcn_readfirstlane(cq.w)};
      uint64_t words[kQuad][WPC];
#pragma unroll
      for (int c = 0; c < kQuad; ++c) {
        const_ptr<uint64_t> bm = bitmap_c + (size_t)cols[c] * WPC;
#pragma unroll
        for (int w = 0; w < WPC; ++w) words[c][w] = bm[w];
      }
      float xv[kQuad][NB];
#pragma unroll
      for (int c = 0; c < kQuad; ++c)
#pragma unroll
        for (int b = 0; b < NB; ++b) xv[c][b] = half_bits_to_float(xs_l[(i * kBatch + u0 + c) * NB + b]);
      // 3. bitmap decode: a row's value sits at the MaskedPopcount of its word
      // below the lane, plus the popcounts of the column's earlier words
      uint32_t vb[kQuad][WPC];
#pragma unroll
      for (int c = 0; c < kQuad; ++c) {
        const uint16_t* slot = reinterpret_cast<const uint16_t*>(val_buf + (u0 + c) * kSlotBytes);
        uint32_t prefix = 0;
#pragma unroll
        for (int w = 0; w < WPC; ++w) {
          vb[c][w] = slot[prefix + mbcnt64(words[c][w])];
          prefix += (uint32_t)__builtin_popcountll(words[c][w]);
        }
      }
      // 4. accumulate where the bitmap bit is set (the word is the lane mask;
      // the compiler turns this into an FMA plus a select on it, which
      // measures faster than branching on EXEC)
#pragma unroll
      for (int c = 0; c < kQuad; ++c)
#pragma unroll
        for (int w = 0; w < WPC; ++w) {
          if (__builtin_amdgcn_inverse_ballot_w64(words[c][w])) {
            const float v = half_bits_to_float(vb[c][w]);
#pragma unroll
            for (int b = 0; b < NB; ++b) acc[w][b] = __builtin_fmaf(v, xv[c][b], acc[w][b]);
          }
        }
    }
  };

  // Two-stage ping-pong: buffer 0 holds even batches, buffer 1 odd ones.
  if (n_batches > 0) issue(0, my_val0, my_bm0);
  for (int i = 0; i < n_batches; i += 2) {
    if (i + 1 < n_batches) {
      issue(i + 1, my_val1, my_bm1);
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(kLoadsPerBatch));
    } else {
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    }
    __builtin_amdgcn_wave_barrier();
    decode(i, my_val0);
    if (i + 1 >= n_batches) break;
    if (i + 2 < n_batches) {
      issue(i + 2, my_val0, my_bm0);
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(kLoadsPerBatch));
    } else {
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    }
    __builtin_amdgcn_wave_barrier();
    decode(i + 1, my_val1);
  }

  // ---- 5. reduce the 4 waves in LDS, write this segment's partial sums
  const int mpad = a.n_stripes * a.tile_m;
  float* red = reinterpret_cast<float*>(val0);
  constexpr int kSlice = Smem<NB>::kSlice;
#pragma unroll
  for (int b0 = 0; b0 < NB; b0 += kSlice) {
    __syncthreads();
#pragma unroll
    for (int w = 0; w < WPC; ++w)
#pragma unroll
      for (int bb = 0; bb < kSlice; ++bb) red[(wave * kSlice + bb) * 256 + 64 * w + lane] = acc[w][b0 + bb];
    __syncthreads();
    const int row = threadIdx.x;
    if (row < 64 * WPC) {
#pragma unroll
      for (int bb = 0; bb < kSlice; ++bb) {
        const int b = b0 + bb;
        if (b < a.batch) {
          float s = 0.0f;
#pragma unroll
          for (int wv = 0; wv < kWaves; ++wv) s += red[(wv * kSlice + bb) * 256 + row];
          // device-coherent store: read back below by whichever workgroup
          // of this stripe arrives last, possibly on another XCD
          __hip_atomic_store(&a.partials[((size_t)seg * a.batch + b) * mpad + (size_t)r * a.tile_m + row],
                             s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
  }

  // ---- split-K completion. The partial stores above bypass the per-XCD L2
  // (device-scope atomics), so waiting for their completion before counting
  // in publishes them without an L2-wide write-back; the last workgroup reads
  // them with device-scope loads.
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t prev = __hip_atomic_fetch_add(&a.counters[r], 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev == (uint32_t)(a.segments - 1));
  }
  __syncthreads();
  if (!s_last) return;
  const int row = threadIdx.x;
  const int m = r * a.tile_m + row;
  if (row < 64 * WPC && m < a.rows) {
    // All segments' partials of a token are requested before any is added, so
    // the reduction costs one memory round trip per kFinal segments, and the
    // sum runs in segment order (deterministic).
    constexpr int kFinal = 32;
    for (int b = 0; b < a.batch; ++b) {
      float s = 0.0f;
      for (int sg0 = 0; sg0 < a.segments; sg0 += kFinal) {
        float v[kFinal];
#pragma unroll
        for (int j = 0; j < kFinal; ++j) {
          const int sg = min(sg0 + j, a.segments - 1);
          v[j] = __hip_atomic_load(&a.partials[((size_t)sg * a.batch + b) * mpad + m], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
#pragma unroll
        for (int j = 0; j < kFinal; ++j)
          if (sg0 + j < a.segments) s += v[j];
      }
      a.y[(size_t)b * a.rows + m] = __half_as_ushort(__float2half_rn(s));
    }
  }
  if (threadIdx.x == 0) __hip_atomic_store(&a.counters[r], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

using spdp::fail;

int hip_fail(hipError_t e, const char* what) {
  return fail(SPDP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Split-K heuristic: about 2048 waves (8 per CU on 256 CUs), every wave
// covering a multiple of 16 columns and at most kMaxWaveCols of them.
// SPDP_SPLITK overrides the number of segments (for tuning).
void choose_split(const spdp_matrix* m, int* segments, int* wave_cols) {
  const int64_t cols = m->cols;
  const int64_t stripes = std::max<int64_t>(1, m->n_stripes);
  int64_t want = std::max<int64_t>(1, 2048 / (kWaves * stripes));
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
  hipError_t e = hipMalloc(&m->d_partials, need * sizeof(float));
  if (e != hipSuccess) {
    m->d_partials = nullptr;
    return e == hipErrorOutOfMemory ? fail(SPDP_ERR_OOM, "hipMalloc of the split-K workspace failed")
                                    : hip_fail(e, "hipMalloc");
  }
  m->partial_floats = need;
  return SPDP_OK;
}

void release_device(spdp_matrix* m) {
  if (m->device < 0) return;
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(m->device);
  (void)hipDeviceSynchronize();
  void* ptrs[] = {m->d_tile_offset, m->d_col_info, m->d_bitmap, m->d_values,
                  m->d_partials, m->d_counters};
  for (void* p : ptrs)
    if (p) (void)hipFree(p);
  m->d_tile_offset = m->d_col_info = m->d_bitmap = m->d_values = nullptr;
  m->d_partials = nullptr;
  m->d_counters = nullptr;
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
    e = hipMalloc(&m->d_counters, (size_t)m->n_stripes * sizeof(uint32_t));
    if (e != hipSuccess) {
      m->d_counters = nullptr;
      st = hip_fail(e, "hipMalloc");
    } else {
      e = hipMemset(m->d_counters, 0, (size_t)m->n_stripes * sizeof(uint32_t));
      if (e != hipSuccess) st = hip_fail(e, "hipMemset");
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
  args.counters = h->d_counters;
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
