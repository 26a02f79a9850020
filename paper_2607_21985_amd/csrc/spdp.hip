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
constexpr int kMaxWords = 4;              // tile_m <= 256
constexpr int kBatchCols = 4;             // active columns staged per wave per round
constexpr int kSlotBytes = 64 * kMaxWords * 2;  // one column of one stripe, fp16
constexpr int kStageBytes = kWaves * kBatchCols * kSlotBytes;  // 16 KiB
constexpr int kMaxBatch = 32;

struct KernelArgs {
  const uint32_t* __restrict__ tile_offset;
  const uint32_t* __restrict__ col_info;
  const uint64_t* __restrict__ bitmap;
  const uint16_t* __restrict__ values;
  const uint16_t* __restrict__ x;
  uint16_t* __restrict__ y;
  float* __restrict__ partials;  // [segments][batch][n_stripes * tile_m]
  uint32_t* __restrict__ counters;  // [n_stripes]
  int rows, cols;
  int tile_m, wpc, tk_log2, n_colblocks, n_stripes;
  int batch;
  int code;       // threshold code: active iff code < (x & 0x7fff) <= 0x7c00
  int wave_cols;  // columns per wave (multiple of 16)
  int segments;   // workgroups per row stripe
};

__device__ __forceinline__ uint32_t mbcnt64(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return __half2float(__ushort_as_half((unsigned short)h));
}

struct Words4 {
  uint64_t w[kMaxWords];
};

template <int NB>
struct Smem {
  static constexpr int kXBytes = kWaves * 64 * NB * 2;   // masked x, fp16 bits
  static constexpr int kSlice = NB < 8 ? NB : 8;          // tokens per reduction pass
  static constexpr int kRedBytes = kWaves * kSlice * 256 * 4;
  static constexpr int kMain = kStageBytes + kXBytes;
  static constexpr int kBytes = kMain > kRedBytes ? kMain : kRedBytes;
};

// Read-only metadata is reached through constant-address-space pointers so
// that uniform (per-column) accesses compile to scalar loads.
template <class T>
using const_ptr = const __attribute__((address_space(4))) T*;

template <class T>
__device__ __forceinline__ const_ptr<T> as_const(const T* p) {
  return reinterpret_cast<const_ptr<T>>(reinterpret_cast<uintptr_t>(p));
}

__device__ __forceinline__ void lds_dma16(const void* src, void* lds_base) {
  __builtin_amdgcn_global_load_lds(src, reinterpret_cast<__attribute__((address_space(3))) void*>(
                                            reinterpret_cast<uintptr_t>(lds_base)),
                                   16, 0, 0);
}

template <int NB>
__global__ __launch_bounds__(kThreads) void spmspv_kernel(KernelArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char smem[Smem<NB>::kBytes];
  __shared__ int s_last;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int seg = blockIdx.x;
  const int r = blockIdx.y;
  const int tk_mask = (1 << a.tk_log2) - 1;
  const int wpc = a.wpc;
  const_ptr<uint32_t> col_info = as_const(a.col_info);
  const_ptr<uint32_t> tile_offset = as_const(a.tile_offset);
  const_ptr<uint64_t> bitmap = as_const(a.bitmap);

  unsigned char* stage = smem + wave * (kBatchCols * kSlotBytes);
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem + kStageBytes) + wave * 64 * NB;

  float acc[kMaxWords][NB];
#pragma unroll
  for (int w = 0; w < kMaxWords; ++w)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[w][b] = 0.0f;

  const int k_begin = (seg * kWaves + wave) * a.wave_cols;
  const int k_end = min(k_begin + a.wave_cols, a.cols);
  const int g_row = r * a.n_colblocks;

  for (int k0 = k_begin; k0 < k_end; k0 += 64) {
    // ---- 1. activity of 64 columns, union over the batch ----
    const int k = k0 + lane;
    const bool in_range = k < k_end;
    uint64_t act = 0;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      uint32_t xb = 0;
      if (in_range && b < a.batch) xb = a.x[(size_t)b * a.cols + k];
      const int mag = (int)(xb & 0x7FFFu);
      const bool on = in_range && b < a.batch && mag > a.code && mag <= 0x7C00;
      act |= __builtin_amdgcn_ballot_w64(on);
      xs[lane * NB + b] = on ? (uint16_t)xb : (uint16_t)0;
    }

    while (act) {
      // ---- 2. pop up to kBatchCols active columns (scalar), fetch metadata ----
      int kc[kBatchCols];
      bool live[kBatchCols];
#pragma unroll
      for (int u = 0; u < kBatchCols; ++u) {
        live[u] = act != 0;
        kc[u] = live[u] ? (int)__builtin_ctzll(act) : 0;  // dead slots alias column k0
        act &= act - 1;
      }
      // Issue every scalar load of the batch before using any result: scalar
      // loads return out of order, so each first use waits for all of them.
      uint32_t ci[kBatchCols], to[kBatchCols];
      Words4 bw[kBatchCols];
#pragma unroll
      for (int u = 0; u < kBatchCols; ++u) {
        const int kk = k0 + kc[u];
        const int g = g_row + (kk >> a.tk_log2);
        const size_t col = ((size_t)g << a.tk_log2) + (kk & tk_mask);
        ci[u] = col_info[col];
        to[u] = tile_offset[g];
        const_ptr<uint64_t> bm = bitmap + col * wpc;  // arrays carry tail padding
#pragma unroll
        for (int w = 0; w < kMaxWords; ++w) bw[u].w[w] = bm[w];
      }
      int base[kBatchCols], nch[kBatchCols];
#pragma unroll
      for (int u = 0; u < kBatchCols; ++u) {
        base[u] = (int)(to[u] + (ci[u] >> 16));
        nch[u] = (int)(((ci[u] & 0xFFFFu) + 7u) >> 3) & -(int)live[u];
      }
      // ---- values: two columns per 16-byte-per-lane load, straight into LDS ----
      const int hsel = lane >> 5;
      const int q = lane & 31;
#pragma unroll
      for (int pr = 0; pr < kBatchCols / 2; ++pr) {
        // Lanes past the column's last chunk re-read its first chunk (same
        // cache line, no extra HBM traffic); what they leave in the slot is
        // never read, because only rows whose bitmap bit is set use a value.
        const int my_base = hsel ? base[2 * pr + 1] : base[2 * pr];
        const int my_nch = hsel ? nch[2 * pr + 1] : nch[2 * pr];
        const int chunk = q < my_nch ? q : 0;
        lds_dma16(a.values + (size_t)my_base + 8 * chunk, stage + 2 * pr * kSlotBytes);
      }
      uint64_t words[kBatchCols][kMaxWords];
#pragma unroll
      for (int u = 0; u < kBatchCols; ++u) {
        const uint64_t keep = 0ull - (uint64_t)live[u];
#pragma unroll
        for (int w = 0; w < kMaxWords; ++w)
          words[u][w] = bw[u].w[w] & keep & (0ull - (uint64_t)(w < wpc));
      }
      __builtin_amdgcn_s_waitcnt(0);  // LDS DMA of this batch has landed
      __builtin_amdgcn_wave_barrier();

      // ---- 3. bitmap decode: rank by masked popcount, read the value ----
      uint32_t vbits[kBatchCols][kMaxWords];
#pragma unroll
      for (int u = 0; u < kBatchCols; ++u) {
        const uint16_t* slot = reinterpret_cast<const uint16_t*>(stage + u * kSlotBytes);
        uint32_t prefix = 0;
#pragma unroll
        for (int w = 0; w < kMaxWords; ++w) {
          const uint32_t rank = min(prefix + mbcnt64(words[u][w]), 255u);
          vbits[u][w] = slot[rank];
          prefix += (uint32_t)__builtin_popcountll(words[u][w]);
        }
      }
      // ---- 4. accumulate where the bitmap bit is set ----
#pragma unroll
      for (int u = 0; u < kBatchCols; ++u) {
        float xv[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) xv[b] = half_bits_to_float(xs[kc[u] * NB + b]);
#pragma unroll
        for (int w = 0; w < kMaxWords; ++w) {
          if (__builtin_amdgcn_inverse_ballot_w64(words[u][w])) {
            const float v = half_bits_to_float(vbits[u][w]);
#pragma unroll
            for (int b = 0; b < NB; ++b) acc[w][b] = __builtin_fmaf(v, xv[b], acc[w][b]);
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }

  // ---- 5. reduce the 4 waves in LDS, write this segment's partial sums ----
  const int mpad = a.n_stripes * a.tile_m;
  float* red = reinterpret_cast<float*>(smem);
  constexpr int kSlice = Smem<NB>::kSlice;
#pragma unroll
  for (int b0 = 0; b0 < NB; b0 += kSlice) {
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kMaxWords; ++w)
#pragma unroll
      for (int bb = 0; bb < kSlice; ++bb)
        if (w < wpc) red[(wave * kSlice + bb) * 256 + 64 * w + lane] = acc[w][b0 + bb];
    __syncthreads();
    const int row = threadIdx.x;
    if (row < a.tile_m) {
#pragma unroll
      for (int bb = 0; bb < kSlice; ++bb) {
        const int b = b0 + bb;
        if (b < a.batch) {
          float s = 0.0f;
#pragma unroll
          for (int wv = 0; wv < kWaves; ++wv) s += red[(wv * kSlice + bb) * 256 + row];
          a.partials[((size_t)seg * a.batch + b) * mpad + (size_t)r * a.tile_m + row] = s;
        }
      }
    }
  }

  // ---- split-K completion: the last workgroup of the stripe finishes Y ----
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t prev = __hip_atomic_fetch_add(&a.counters[r], 1u, __ATOMIC_ACQ_REL,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev == (uint32_t)(a.segments - 1));
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  const int row = threadIdx.x;
  const int m = r * a.tile_m + row;
  if (row < a.tile_m && m < a.rows) {
    for (int b = 0; b < a.batch; ++b) {
      float s = 0.0f;
      for (int sg = 0; sg < a.segments; ++sg)
        s += a.partials[((size_t)sg * a.batch + b) * mpad + m];
      a.y[(size_t)b * a.rows + m] = __half_as_ushort(__float2half_rn(s));
    }
  }
  if (threadIdx.x == 0) a.counters[r] = 0u;
}

using spdp::fail;

int hip_fail(hipError_t e, const char* what) {
  return fail(SPDP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Split-K heuristic: aim for about 1024 workgroups (4 per CU on 256 CUs)
// while giving every wave at least 16 columns; SPDP_SPLITK overrides the
// number of segments for tuning.
void choose_split(const spdp_matrix* m, int* segments, int* wave_cols) {
  const int64_t cols = m->cols;
  int64_t want = std::max<int64_t>(1, 1024 / std::max<int64_t>(1, m->n_stripes));
  if (const char* env = std::getenv("SPDP_SPLITK")) {
    const long v = std::strtol(env, nullptr, 10);
    if (v >= 1) want = v;
  }
  const int64_t max_seg = std::max<int64_t>(1, (cols + kWaves * 16 - 1) / (kWaves * 16));
  const int64_t s = std::min(want, max_seg);
  int64_t wc = (cols + s * kWaves - 1) / (s * kWaves);
  wc = (wc + 15) / 16 * 16;
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

template <int NB>
hipError_t launch(const KernelArgs& args, dim3 grid, hipStream_t stream) {
  hipLaunchKernelGGL(spmspv_kernel<NB>, grid, dim3(kThreads), 0, stream, args);
  return hipGetLastError();
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
  args.wpc = h->tile_m / 64;
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
    e = launch<1>(args, grid, s);
  else if (batch <= 2)
    e = launch<2>(args, grid, s);
  else if (batch <= 4)
    e = launch<4>(args, grid, s);
  else if (batch <= 8)
    e = launch<8>(args, grid, s);
  else if (batch <= 16)
    e = launch<16>(args, grid, s);
  else
    e = launch<32>(args, grid, s);
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return SPDP_OK;
}

void spdp_free(spdp_handle_t h) {
  if (!h) return;
  release_device(h);
  delete h;
}

}  // extern "C"
