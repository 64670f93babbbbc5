// A chain of GEMVs in one persistent launch: the products of a decode step run in
// order, each after the previous one has finished (a grid-wide barrier between
// consecutive products), so the output of one can be the input of any later one.
// Decoding is memory-bound (Section 2.4): a separate launch per product costs a
// dispatch and a ramp of the memory pipeline each time, which a chain of a
// hundred small products pays a hundred times. Here every block stays resident;
// between products a block only waits for the others at the barrier, and it
// loads the codes of its first rows of the next product before it waits, since
// the weights do not depend on the previous output.
//
// Work split: for K = 128*32 a wave takes two rows (32 lanes, one chunk each);
// for 32 < C <= 88 chunks a wave takes one row, lane l the chunks l and l + 64.
// (One kernel serves every format, so the format with the largest items sets the
// register budget of all; that is why a lane holds one item ahead, not two.)
// Waves walk the rows of a product grid-stride. The block stages x in LDS once
// per product. Rows are reduced in registers with DPP, so results are
// deterministic and equal, row for row, from run to run.
#include "gemv_common.h"

namespace qx {

constexpr int kChainThreads = 256;
constexpr int kChainWaves = kChainThreads / 64;

namespace {

// Workspace header (QX_CHAIN_HEADER_BYTES): the words below, the release flag at
// byte 128 and one arrival counter per block group at 256 + 64*g, each on its own
// 64-byte line.
struct ChainHeader {
  uint32_t arrive;  // groups arrived at barriers in this launch
  uint32_t done;    // blocks that finished
  uint32_t error;   // nonzero: a barrier wait gave up, or the launch did not match the table
  uint32_t count;   // products in the table
  uint32_t plan;    // kernel variant chosen when the table was written
};
constexpr int kGroups = 32;
constexpr int kFlagWord = 128 / 4;
constexpr int kGroupWord0 = 256 / 4, kGroupStride = 64 / 4;

__device__ __forceinline__ uint32_t load_relaxed(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Grid-wide barrier number b (1, 2, ...). Outputs are written with device-scope
// stores and inputs staged with device-scope loads (both bypass the caches that
// are not coherent across the chip), so the barrier needs no cache write-back or
// invalidation: each wave waits for its own stores to complete, one thread per
// block adds to its group's counter, the last block of a group adds to the
// group total, and the last group raises the flag to b. (With device-scope
// fences instead, a barrier measured 16 to 53 us on 512 blocks; this one 2 us.)
// Returns false, and flags the error, once spin_limit polls have found the flag
// low or another block has flagged one, so that every wave always exits.
__device__ __forceinline__ bool grid_barrier(uint32_t* hw, uint32_t b, uint32_t spin_limit, int* ok) {
  __builtin_amdgcn_s_waitcnt(0);  // this wave's stores are complete
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t G = gridDim.x, grp = blockIdx.x % kGroups;
    const uint32_t gsize = (G - grp + kGroups - 1) / kGroups, ngroups = G < kGroups ? G : kGroups;
    const uint32_t old =
        __hip_atomic_fetch_add(hw + kGroupWord0 + grp * kGroupStride, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == b * gsize - 1) {
      const uint32_t o2 = __hip_atomic_fetch_add(hw, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (o2 == b * ngroups - 1) __hip_atomic_store(hw + kFlagWord, b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    uint32_t polls = 0;
    int good = 1;
    while (load_relaxed(hw + kFlagWord) < b) {
      if (load_relaxed(hw + 2) != 0 || ++polls >= spin_limit) {
        __hip_atomic_store(hw + 2, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        good = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    *ok = good;
  }
  __syncthreads();
  return *ok != 0;
}

// x pieces of a product, read with device-scope loads (an earlier product of
// the chain may have written them on another part of the chip).
template <int XP>
__device__ __forceinline__ void load_x_coherent(const uint16_t* __restrict__ x, int ct, u32x4 (&xr)[XP]) {
  const uint32_t* src = reinterpret_cast<const uint32_t*>(x);
#pragma unroll
  for (int i = 0; i < XP; ++i) {
    const int p = min((int)threadIdx.x + i * kChainThreads, ct * 16 - 1);
    xr[i].x = load_relaxed(src + 4 * p);
    xr[i].y = load_relaxed(src + 4 * p + 1);
    xr[i].z = load_relaxed(src + 4 * p + 2);
    xr[i].w = load_relaxed(src + 4 * p + 3);
  }
}

__device__ __forceinline__ void store_y(uint16_t* y, int row, float v) {
  __hip_atomic_store(y + row, (uint16_t)float_to_half_bits(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The first item of a wave's unit of work: for C == 32 the lane's chunk of one of
// the wave's two rows; else chunk `lane` of the wave's row (chunk lane + 64, if
// any, is loaded while the unit is finished, to keep registers for occupancy).
template <int BITS, int KIND, int G>
__device__ __forceinline__ void load_unit(Item<BITS, KIND, G>& it, const char* packed, size_t meta_off,
                                          int n, int C, int unit, int lane) {
  const int G_row = C * 128 / G;
  if (C == 32)
    load_item<BITS, KIND, G>(it, packed, meta_off, min(2 * unit + (lane >> 5), n - 1), lane & 31, 32, 32 * 128 / G);
  else
    load_item<BITS, KIND, G>(it, packed, meta_off, unit, min(lane, C - 1), C, G_row);
}

// One product: stage x, then the wave's units grid-stride. `first` holds the
// first unit of the wave, loaded before the barrier that precedes the product.
// C32: the product has K = 128*32 (two rows per wave), else 32 < C <= 88 (one).
template <int BITS, int KIND, int G, bool C32>
__device__ __forceinline__ void run_product(char* ws, const ChainOp& op, char* xs, float2* gs,
                                            const Item<BITS, KIND, G>& first, int unit0, int stride) {
  constexpr int NG = 128 / G;
  constexpr int XP = C32 ? 32 * 16 / kChainThreads : (kMaxTileChunks * 16 + kChainThreads - 1) / kChainThreads;
  const int n = op.desc.n, k = C32 ? 32 * 128 : op.desc.k, C = k >> 7;
  const char* packed = ws + op.packed;
  const uint16_t* x = reinterpret_cast<const uint16_t*>(ws + op.x);
  uint16_t* y = reinterpret_cast<uint16_t*>(ws + op.y);
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int lane = threadIdx.x & 63;
  const int units = C32 ? (n + 1) / 2 : n;
  const DecodeConsts kc = decode_consts();

  u32x4 xr[XP];
  load_x_coherent<XP>(x, C, xr);
  store_x<BITS, KIND, G, XP, C32>(xr, C, xs, gs, kChainThreads);
  __syncthreads();
  for (int u = unit0; u < units; u += stride) {
    Item<BITS, KIND, G> it;
    if (u == unit0) it = first;
    else if (C32) load_item<BITS, KIND, G>(it, packed, meta_off, min(2 * u + (lane >> 5), n - 1), lane & 31, 32, 32 * 128 / G);
    else load_item<BITS, KIND, G>(it, packed, meta_off, u, min(lane, C - 1), C, k / G);
    // x is the same for every unit; an opaque offset keeps the compiler from
    // hoisting its LDS reads out of the loop into registers (up to 128 per lane),
    // which would cost more occupancy than the reads cost LDS bandwidth
    int opaque = 0;
    asm volatile("" : "+v"(opaque));
    const char* xl = xs + opaque;
    if (C32) {
      const int c = lane & 31, row = 2 * u + (lane >> 5);
      float v = chunk_dot<BITS, KIND, G>(it, xl + c * kXBlock, gs + c * NG, kc);
      v = half_wave_sum(v);
      if (c == 31 && row < n) store_y(y, row, v);
    } else {
      Item<BITS, KIND, G> it2;
      if (C > 64) load_item<BITS, KIND, G>(it2, packed, meta_off, u, min(lane + 64, C - 1), C, k / G);
      float v = 0.f;
      if (lane < C) v = chunk_dot<BITS, KIND, G>(it, xl + lane * kXBlock, gs + lane * NG, kc);
      if (C > 64 && lane + 64 < C)
        v += chunk_dot<BITS, KIND, G>(it2, xl + (lane + 64) * kXBlock, gs + (lane + 64) * NG, kc);
      v = wave_sum(v);
      if (lane == 63) store_y(y, u, v);
    }
  }
}

// A product's path: its format and whether K = 128*32. Path ids (0..23) are
// ((bits - 3)*2 + kind)*6 + log2(group/32)*2 + (K == 128*32); the host writes each
// product's id in its descriptor's flags word.
constexpr int path_bits(int id) { return 3 + id / 12; }
constexpr int path_kind(int id) { return (id / 6) % 2; }
constexpr int path_group(int id) { return 32 << ((id / 2) % 3); }
constexpr bool path_c32(int id) { return id % 2 == 1; }
template <int ID>
using PathItem = Item<path_bits(ID), path_kind(ID), path_group(ID)>;
template <int ID>
constexpr int path_dwords() { return (int)(sizeof(PathItem<ID>) / 4); }

template <uint32_t MASK, int ID = 0>
constexpr int max_path_dwords() {
  if constexpr (ID == 24) {
    return 1;
  } else {
    constexpr int here = ((MASK >> ID) & 1u) ? path_dwords<ID>() : 1;
    constexpr int rest = max_path_dwords<MASK, ID + 1>();
    return here > rest ? here : rest;
  }
}

template <typename T, int N>
__device__ __forceinline__ void to_raw(const T& it, uint32_t (&raw)[N]) {
  static_assert(sizeof(T) <= 4 * N, "raw buffer too small");
  const uint32_t* w = reinterpret_cast<const uint32_t*>(&it);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) raw[i] = w[i];
}
template <typename T, int N>
__device__ __forceinline__ void from_raw(T& it, const uint32_t (&raw)[N]) {
  uint32_t* w = reinterpret_cast<uint32_t*>(&it);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) w[i] = raw[i];
}

// Loads the first unit of product `op` (path `id`) into raw; false if the path
// is not compiled into this kernel.
template <uint32_t MASK, int N, int ID = 0>
__device__ __forceinline__ bool prefetch_path(int id, char* ws, const ChainOp& op, uint32_t (&raw)[N], int gw) {
  if constexpr (ID == 24) {
    return false;
  } else {
    if constexpr ((MASK >> ID) & 1u) {
      if (id == ID) {
        constexpr int B = path_bits(ID);
        const int n = op.desc.n, C = op.desc.k >> 7;
        if (gw < (path_c32(ID) ? (n + 1) / 2 : n)) {
          PathItem<ID> it;
          load_unit<B, path_kind(ID), path_group(ID)>(it, ws + op.packed, (size_t)n * op.desc.k * B / 8, n, C, gw,
                                                      threadIdx.x & 63);
          to_raw(it, raw);
        }
        return true;
      }
    }
    return prefetch_path<MASK, N, ID + 1>(id, ws, op, raw, gw);
  }
}

template <uint32_t MASK, int N, int ID = 0>
__device__ __forceinline__ bool run_path(int id, char* ws, const ChainOp& op, char* xs, float2* gs,
                                         const uint32_t (&raw)[N], int gw, int stride) {
  if constexpr (ID == 24) {
    return false;
  } else {
    if constexpr ((MASK >> ID) & 1u) {
      if (id == ID) {
        PathItem<ID> it;
        from_raw(it, raw);
        run_product<path_bits(ID), path_kind(ID), path_group(ID), path_c32(ID)>(ws, op, xs, gs, it, gw, stride);
        return true;
      }
    }
    return run_path<MASK, N, ID + 1>(id, ws, op, xs, gs, raw, gw, stride);
  }
}

// The chain, for the paths in MASK (one kernel per set of paths, so that a chain
// of light formats does not pay the registers of the heaviest one). Each block:
// load the first unit of product 0; then per product: run it, load the first
// unit of the next one, wait at the barrier.
template <uint32_t MASK>
__global__ __launch_bounds__(kChainThreads) void chain_kernel(char* __restrict__ ws, int count,
                                                              uint32_t plan, uint32_t spin_limit) {
  constexpr int N = max_path_dwords<MASK>();
  __shared__ __align__(16) char xs[kMaxTileChunks * kXBlock];
  __shared__ float2 gs[kMaxTileChunks * 4];
  __shared__ int ok;
  ChainHeader* h = reinterpret_cast<ChainHeader*>(ws);
  const ChainOp* ops = reinterpret_cast<const ChainOp*>(ws + QX_CHAIN_HEADER_BYTES);
  const int gw = blockIdx.x * kChainWaves + (threadIdx.x >> 6), stride = gridDim.x * kChainWaves;
  bool good = h->count == (uint32_t)count && h->plan == plan;
  uint32_t raw[N];
  if (good) good = prefetch_path<MASK>((int)ops[0].desc.flags, ws, ops[0], raw, gw);
  for (int s = 0; good && s < count; ++s) {
    good = run_path<MASK>((int)ops[s].desc.flags, ws, ops[s], xs, gs, raw, gw, stride);
    if (!good || s + 1 == count) break;
    // the next product's weights do not depend on this one's output
    good = prefetch_path<MASK>((int)ops[s + 1].desc.flags, ws, ops[s + 1], raw, gw);
    if (good) good = grid_barrier(reinterpret_cast<uint32_t*>(ws), (uint32_t)(s + 1), spin_limit, &ok);
  }
  if (threadIdx.x == 0) {
    if (!good) __hip_atomic_store(&h->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // the last block to finish rearms the barrier for the next launch
    const uint32_t prev = __hip_atomic_fetch_add(&h->done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (good && prev == gridDim.x - 1) {
      uint32_t* hw = reinterpret_cast<uint32_t*>(ws);
      for (int g = 0; g < kGroups; ++g)
        __hip_atomic_store(hw + kGroupWord0 + g * kGroupStride, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(hw + kFlagWord, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&h->arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&h->done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Path sets with a kernel each: every path; the decoder mix of 3-bit codebook
// and 4-bit uniform, groups of 128 (attention with K = 128*32, MLP of any K);
// and each single format (both K classes).
constexpr uint32_t kAllPaths = 0xFFFFFFu;
constexpr uint32_t kDecoderPaths = (1u << 11) | (1u << 10) | (1u << 17) | (1u << 16);

template <uint32_t MASK>
int launch_mask(void* ws, int count, uint32_t plan, uint32_t spin_limit, hipStream_t s) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, chain_kernel<MASK>, kChainThreads, 0) != hipSuccess ||
      per_cu < 1)
    return QX_E_HIP;
  char* w = static_cast<char*>(ws);
  void* args[] = {&w, &count, &plan, &spin_limit};
  const dim3 grid((unsigned)(cus * per_cu)), block(kChainThreads);
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(chain_kernel<MASK>), grid, block, args, 0, s) ==
                 hipSuccess
             ? QX_OK
             : QX_E_HIP;
}

}  // namespace

int chain_path(const qx_desc* d) {
  const int gi = d->group == 32 ? 0 : d->group == 64 ? 1 : 2;
  return ((d->bits - 3) * 2 + d->kind) * 6 + gi * 2 + (d->k == 32 * 128 ? 1 : 0);
}

bool chain_op_supported(const qx_desc* d) {
  const int C = d->k / 128;
  return d->kind != QX_Q4X && (C == 32 || (C > 32 && C <= kMaxTileChunks));
}

// Plans: 0 = every path, 1 = decoder mix, 2 + f = format f alone (f = path / 2).
uint32_t chain_plan(uint32_t paths) {
  if ((paths & ~kDecoderPaths) == 0) return 1;
  for (uint32_t f = 0; f < 12; ++f)
    if ((paths & ~(3u << (2 * f))) == 0) return 2 + f;
  return 0;
}

int launch_chain(void* ws, int count, uint32_t plan, uint32_t spin_limit, hipStream_t s) {
  switch (plan) {
#define QX_CHAIN_FMT(F) \
  case 2 + F: return launch_mask<(3u << (2 * F))>(ws, count, plan, spin_limit, s);
    QX_CHAIN_FMT(0) QX_CHAIN_FMT(1) QX_CHAIN_FMT(2) QX_CHAIN_FMT(3) QX_CHAIN_FMT(4) QX_CHAIN_FMT(5)
    QX_CHAIN_FMT(6) QX_CHAIN_FMT(7) QX_CHAIN_FMT(8) QX_CHAIN_FMT(9) QX_CHAIN_FMT(10) QX_CHAIN_FMT(11)
#undef QX_CHAIN_FMT
    case 1: return launch_mask<kDecoderPaths>(ws, count, plan, spin_limit, s);
    case 0: return launch_mask<kAllPaths>(ws, count, plan, spin_limit, s);
    default: return QX_E_ARG;
  }
}

static_assert(256 + kGroups * 64 <= QX_CHAIN_HEADER_BYTES, "chain header too small");

}  // namespace qx
