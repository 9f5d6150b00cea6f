// Fused tile-parallel EntroPack decode for gfx950 (Section 3.7): host side and
// the kernels of prepared stacks, the fused products and the table images.
// The device code and its description are in decode_kernels.h.
#include "decode_kernels.h"
#include "decode_launch.h"

namespace ep {
namespace {

// Clears Y before the launches that add partial sums to it.  A kernel rather
// than hipMemsetAsync, so that a caller may capture the call in a graph.
__global__ void zero_i32_kernel(int32_t* __restrict__ y, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    gptr<int32_t>(y)[i] = 0;
}

// ---- host side ---------------------------------------------------------------------
bool clear_i32(int32_t* y, int64_t count, hipStream_t s) {
  if (count <= 0) return true;
  const unsigned blocks = (unsigned)std::min<int64_t>((count + 255) / 256, 4096);
  hipLaunchKernelGGL(zero_i32_kernel, dim3(blocks), dim3(256), 0, s, y, count);
  return hipGetLastError() == hipSuccess;
}

struct DeviceProps {
  int cus = 0;
  size_t max_lds = 0;
};

DeviceProps device_props() {
  static std::mutex mu;
  static std::vector<DeviceProps> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DeviceProps{};
  std::lock_guard<std::mutex> g(mu);
  if ((int)cache.size() <= dev) cache.resize(dev + 1);
  if (!cache[dev].cus) {
    int cus = 0, lds = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 0;
    if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) lds = 0;
    cache[dev].cus = cus;
    cache[dev].max_lds = (size_t)lds;
  }
  return cache[dev];
}

uint32_t lds_bytes(uint32_t path, const ep_tensor_info& I) {
  if (path == kPathGlobal) return global_layout(I.table_A).total + kRingBytes;
  if (path != kPathSearch) return (64u << I.prob_bits) + kRingBytes;
  return search_layout(I.prob_bits, I.sum_alphabet).total + kRingBytes;
}

float dtype_max(int dt) {
  switch (dt) {
    case EP_BF16: return 3.38953139e38f;
    case EP_FP16: return 65504.0f;
    case EP_FP8_E4M3: return 448.0f;
    case EP_FP8_E5M2: return 57344.0f;
    default: return 3.4e38f;
  }
}

bool valid_out_dtype(int dt) {
  return dt == EP_BF16 || dt == EP_FP16 || dt == EP_FP32 || dt == EP_FP8_E4M3 || dt == EP_FP8_E5M2 ||
         dt == EP_INT8 || dt == EP_UINT8 || dt == EP_COORD2_I32;
}

// tables_only: the descriptor only serves a table build (no output, no dequant).
int fill_layer(const ep_tensor_info& I, const void* d_blob, int out_dtype, void* d_out,
               float* d_dequant, uint32_t t0, uint32_t t1, LayerDev& D, bool tables_only = false) {
  if (!d_blob || !d_out) return fail(EP_ERR_ARG, "decode: null device pointer");
  if (I.container && !d_dequant && !tables_only)
    return fail(EP_ERR_ARG, "decode: a container tensor needs d_dequant (its row scales)");
  if (!valid_out_dtype(out_dtype)) return fail(EP_ERR_ARG, "decode: unknown output dtype");
  if (t0 > t1 || t1 > I.n_tiles) return fail(EP_ERR_ARG, "decode: tile range outside the tensor");
  if (!I.rows || !I.cols || I.cols % 8 || I.prob_bits < 9 || I.prob_bits > 15 || !I.tile_vectors)
    return fail(EP_ERR_ARG, "decode: tensor info not filled by ep_blob_info");
  if (!path_fits(I.path, I))
    return fail(EP_ERR_ARG, "decode: the tensor's tables do not fit the decode path in its info");
  std::memset(&D, 0, sizeof D);
  D.path = I.path;
  if (I.path == kPathGlobal) {
    const GlobalLayout G = global_layout(I.table_A);
    D.g_bits = G.g_bits;
    D.g_meta = G.meta;
  }
  D.blob = static_cast<const uint8_t*>(d_blob);
  D.out = d_out;
  D.dequant = d_dequant;
  D.rows = I.rows;
  D.cols = I.cols;
  D.cvec = I.cols / 8;
  D.b = I.prob_bits;
  D.V = I.tile_vectors;
  D.n_tiles = I.n_tiles;
  D.container = I.container;
  D.tile_begin = t0;
  D.tile_end = t1;
  D.tpt = kTilesPerTask;
  D.n_tasks = (t1 - t0 + kTilesPerTask - 1) / kTilesPerTask;
  D.out_dtype = (uint32_t)out_dtype;
  D.saturate = I.max_abs_weight >= dtype_max(out_dtype) ? 1u : 0u;
  D.coset_f0 = I.coset_f0;
  D.coset_f1 = I.coset_f1;
  D.sum_A = I.sum_alphabet;
  const uint64_t pay = (2ull * I.payload_words + 3) / 4 * 4;
  if (pay > 0xFFFFFFF0ull) return fail(EP_ERR_UNSUPPORTED, "decode: payload section above 4 GiB");
  D.pay_bytes = (uint32_t)pay;
  const uint32_t d = D.cvec;
  if ((d & (d - 1)) == 0) {
    D.div_pow2 = 1;
    D.div_shift = 0;
    while ((1u << D.div_shift) < d) D.div_shift++;
  } else {
    uint32_t lg = 0;
    while ((1ull << lg) < d) lg++;
    D.div_pow2 = 0;
    D.div_magic = (uint32_t)(((1ull << 32) * ((1ull << lg) - d)) / d + 1);
    D.div_shift = lg - 1;
  }
  D.off_sigma = I.off_sigma;
  D.off_delta = I.off_delta;
  D.off_states = I.off_states;
  D.off_offsets = I.off_offsets;
  D.off_payload = I.off_payload;
  uint32_t base = 0;
  for (int t = 0; t < 16; t++) {
    D.tab_off[t] = I.table_off[t];
    D.tab_min[t] = I.table_min[t];
    D.tab_A[t] = I.table_A[t];
    D.tab_base[t] = base;
    base += I.table_A[t];
  }
  return EP_OK;
}

// Workgroups of a launch: as many as the CUs hold (one per CU when the tables
// take most of the LDS), but never more than there are tasks.  A small layer
// list is spread over all CUs rather than packed into few workgroups: a task
// is a long serial chain of symbol rounds, so a lightly loaded CU finishes it
// sooner.
uint32_t groups_for(uint32_t path, uint32_t lds, uint32_t tasks, const DeviceProps& P) {
  uint32_t per_cu = path == kPathLut || path == kPathWide || path == kPathMixed
                        ? 1u
                        : (uint32_t)std::max<size_t>(1, std::min<size_t>(2, 160 * 1024 / std::max<uint32_t>(lds, 1)));
  uint32_t g = (uint32_t)P.cus * per_cu;
  return std::max(1u, std::min(g, tasks));
}

}  // namespace

template <int PATH>
int set_lds_limit(size_t bytes) {
  if constexpr (PATH == kPathMixed) {
    return set_mixed_lds_limit(bytes) == hipSuccess ? EP_OK : EP_ERR_HIP;
  } else {
    hipError_t e1 = set_args_lds_limit(PATH, bytes);
    hipError_t e2 = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_ws_kernel<PATH>),
                                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    hipError_t e3 = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_dot_kernel<PATH>),
                                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    return (e1 == hipSuccess && e2 == hipSuccess && e3 == hipSuccess) ? EP_OK : EP_ERR_HIP;
  }
}

bool valid_launch_path(uint32_t path) {
  return path == kPathLut || path == kPathWide || path == kPathSearch || path == kPathGlobal ||
         path == (uint32_t)kPathMixed;
}

// Grid of a launch over `total` tasks: G workgroups of `per` consecutive tasks.
int launch_geometry(uint32_t path, uint32_t total, uint32_t lds, uint32_t& G, uint32_t& per) {
  DeviceProps P = device_props();
  if (!P.cus) return fail(EP_ERR_HIP, "decode: no HIP device");
  if (lds > P.max_lds) return fail(EP_ERR_UNSUPPORTED, "decode: tables exceed the device LDS");
  G = groups_for(path, lds, total, P);
  per = (total + G - 1) / G;
  G = (total + per - 1) / per;
  int rc = path == kPathLut ? set_lds_limit<kPathLut>(lds)
           : path == kPathWide ? set_lds_limit<kPathWide>(lds)
           : path == kPathSearch ? set_lds_limit<kPathSearch>(lds)
           : path == kPathGlobal ? set_lds_limit<kPathGlobal>(lds)
                                 : set_lds_limit<kPathMixed>(lds);
  if (rc) return fail(EP_ERR_HIP, "decode: cannot raise the kernel's LDS limit");
  return EP_OK;
}

// Launch over a descriptor list already in device memory.
int launch_list(uint32_t path, const LayerDev* dl, int n, uint32_t total, uint32_t lds,
                int32_t* d_status, hipStream_t s, const char* who) {
  uint32_t G = 0, per = 0;
  int rc = launch_geometry(path, total, lds, G, per);
  if (rc) return rc;
  if (path == kPathLut)
    hipLaunchKernelGGL(decode_ws_kernel<kPathLut>, dim3(G), dim3(kThreads), lds, s, dl, n, total, per, d_status);
  else if (path == kPathWide)
    hipLaunchKernelGGL(decode_ws_kernel<kPathWide>, dim3(G), dim3(kThreads), lds, s, dl, n, total, per, d_status);
  else if (path == kPathSearch)
    hipLaunchKernelGGL(decode_ws_kernel<kPathSearch>, dim3(G), dim3(kThreads), lds, s, dl, n, total, per, d_status);
  else if (path == kPathGlobal)
    hipLaunchKernelGGL(decode_ws_kernel<kPathGlobal>, dim3(G), dim3(kThreads), lds, s, dl, n, total, per, d_status);
  else
    launch_mixed_ws(dl, n, total, per, G, lds, d_status, s);
  if (hipGetLastError() != hipSuccess) return fail(EP_ERR_HIP, (std::string(who) + ": launch failed").c_str());
  return EP_OK;
}

// Launch the layers of one decode path: by-value descriptors when they fit,
// else from d_ws (copied there first on the same stream).
int launch_layers(uint32_t path, const std::vector<LayerDev>& D, uint32_t total, uint32_t lds,
                  void* d_ws, uint64_t ws_bytes, int32_t* d_status, hipStream_t s,
                  const char* who, bool dot = false) {
  const int n = (int)D.size();
  if (dot && n > kArgLayers) return fail(EP_ERR_ARG, (std::string(who) + ": too many layers").c_str());
  if (n > kArgLayers) {
    if (!d_ws || ws_bytes < sizeof(LayerDev) * (uint64_t)n)
      return fail(EP_ERR_ARG, "ep_decode_layers: workspace too small");
    if (hipMemcpyAsync(d_ws, D.data(), sizeof(LayerDev) * D.size(), hipMemcpyHostToDevice, s) != hipSuccess)
      return fail(EP_ERR_HIP, "ep_decode_layers: descriptor copy failed");
    return launch_list(path, static_cast<const LayerDev*>(d_ws), n, total, lds, d_status, s, who);
  }
  uint32_t G = 0, per = 0;
  int rc = launch_geometry(path, total, lds, G, per);
  if (rc) return rc;
  {
    LayerList list;
    std::memset(&list, 0, sizeof list);
    for (int i = 0; i < n; i++) list.L[i] = D[i];
    if (dot && path == kPathLut)
      hipLaunchKernelGGL(decode_dot_kernel<kPathLut>, dim3(G), dim3(kThreads), lds, s, list, n, total, per, d_status);
    else if (dot && path == kPathWide)
      hipLaunchKernelGGL(decode_dot_kernel<kPathWide>, dim3(G), dim3(kThreads), lds, s, list, n, total, per, d_status);
    else if (dot && path == kPathSearch)
      hipLaunchKernelGGL(decode_dot_kernel<kPathSearch>, dim3(G), dim3(kThreads), lds, s, list, n, total, per, d_status);
    else if (dot)
      hipLaunchKernelGGL(decode_dot_kernel<kPathGlobal>, dim3(G), dim3(kThreads), lds, s, list, n, total, per, d_status);
    else if (path == (uint32_t)kPathMixed)
      launch_mixed_args(&list, n, total, per, G, lds, d_status, s);
    else
      launch_args(path, &list, n, total, per, G, lds, d_status, s);
  }
  if (hipGetLastError() != hipSuccess) return fail(EP_ERR_HIP, (std::string(who) + ": launch failed").c_str());
  return EP_OK;
}

// A launch of fewer four-tile tasks than this runs two-tile tasks (one chain
// per wave) when every layer takes the same slot-table path at b = 11: twice
// as many waves, each issuing half the instructions per symbol (see
// field_step1).  The environment variable EP_SMALL_TASK_LIMIT overrides the
// limit (0: always four-tile tasks).
constexpr uint32_t kSmallLaunchTasks = 2048;

uint32_t small_task_limit() {
  const char* e = std::getenv("EP_SMALL_TASK_LIMIT");
  if (!e || !*e) return kSmallLaunchTasks;
  char* end = nullptr;
  const unsigned long v = std::strtoul(e, &end, 10);
  return (end && *end == 0 && v <= 0xFFFFFFFFul) ? (uint32_t)v : kSmallLaunchTasks;
}

void use_small_tasks(std::vector<LayerDev>& D, uint32_t& total) {
  if (total == 0 || total >= small_task_limit()) return;
  for (const LayerDev& d : D)
    if ((d.path != kPathLut && d.path != kPathWide) || d.path != D[0].path || d.out_dtype == kOutDotI8 ||
        d.b != 11)
      return;
  uint32_t tasks = 0;
  for (LayerDev& d : D) {
    d.tpt = 2;
    d.n_tasks = (d.tile_end - d.tile_begin + 1) / 2;
    d.task_begin = tasks;
    tasks += d.n_tasks;
  }
  total = tasks;
}

int decode_tiles(const ep_tensor_info* info, const void* d_blob, int out_dtype, void* d_out,
                 float* d_dequant, uint32_t t0, uint32_t t1, int32_t* d_status, void* stream) {
  if (!info) return fail(EP_ERR_ARG, "ep_decode_tiles: null info");
  std::vector<LayerDev> D(1);
  int rc = fill_layer(*info, d_blob, out_dtype, d_out, d_dequant, t0, t1, D[0]);
  if (rc) return rc;
  uint32_t total = D[0].n_tasks;
  use_small_tasks(D, total);
  if (total == 0) return EP_OK;
  return launch_layers(info->path, D, total, lds_bytes(info->path, *info), nullptr, 0,
                       d_status, static_cast<hipStream_t>(stream), "ep_decode_tiles");
}

// Fused decode and small-batch product: the INT8 container values of every
// tile, multiplied into X as they are decoded (see lut_task).
int decode_matmul_i8(const ep_tensor_info* info, const void* d_blob, const int8_t* d_x, int m,
                     int32_t* d_y, float* d_dequant, int32_t* d_status, void* stream) {
  if (!info) return fail(EP_ERR_ARG, "ep_decode_matmul_i8: null info");
  if (info->container != EP_CONT_INT8_ROW)
    return fail(EP_ERR_UNSUPPORTED, "ep_decode_matmul_i8: the tensor is not in the INT8 row container");
  if (m < 1 || m > (int)kDotMaxTokens) return fail(EP_ERR_ARG, "ep_decode_matmul_i8: m must be 1 .. 8");
  if (!d_x || !d_y) return fail(EP_ERR_ARG, "ep_decode_matmul_i8: null X or Y");
  if (info->cols > 131071)
    return fail(EP_ERR_UNSUPPORTED, "ep_decode_matmul_i8: rows longer than 131071 weights may overflow int32");
  std::vector<LayerDev> D(1);
  int rc = fill_layer(*info, d_blob, EP_INT8, d_y, d_dequant, 0, info->n_tiles, D[0]);
  if (rc) return rc;
  D[0].out_dtype = kOutDotI8;
  D[0].saturate = 0;
  D[0].x = d_x;
  D[0].m = (uint32_t)m;
  // More than four rows of X: two-tile tasks with one chain per wave, whose
  // eight running sums per lane fit the registers (with two chains they spill).
  if (m > 4 && (D[0].path == kPathLut || D[0].path == kPathWide) && D[0].b == 11) {
    D[0].tpt = 2;
    D[0].n_tasks = (D[0].tile_end - D[0].tile_begin + 1) / 2;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!clear_i32(d_y, (int64_t)m * info->rows, s))
    return fail(EP_ERR_HIP, "ep_decode_matmul_i8: clearing Y failed");
  if (D[0].n_tasks == 0) return EP_OK;
  return launch_layers(info->path, D, D[0].n_tasks, lds_bytes(info->path, *info), nullptr, 0,
                       d_status, s, "ep_decode_matmul_i8", true);
}

// A layer's decode tables as built in LDS (ring_offset bytes, at most this).
constexpr uint64_t kTableImageBytes = 128 * 1024;

// Workspace of the fused MFMA product: the table image that
// ep_decode_gemm_i8_prepare writes, the layer descriptor the table kernel
// reads, then one slab per workgroup.
constexpr uint64_t kGemmDescOffset = kTableImageBytes;
constexpr uint64_t kGemmSlabsOffset = kGemmDescOffset + ((sizeof(LayerDev) + 255) & ~255ull);

// Fused decode and MFMA product: grid, margin rows and slab bytes of a tensor
// (elem: bytes per decoded weight, 1 for the INT8 product, 2 for the BF16 one).
struct GemmGeom {
  uint32_t groups, margin, n_blocks, rows_per_block;
  uint64_t slab_bytes;
};

int gemm_geometry(const ep_tensor_info& I, uint32_t elem, GemmGeom& G) {
  DeviceProps P = device_props();
  if (!P.cus) return fail(EP_ERR_HIP, "ep_decode_gemm: no HIP device");
  const uint32_t cvec = I.cols / 8;
  // rows a block's tiles reach past either side: its tile range is widened to
  // whole tasks of kTilesPerTask tiles
  G.margin = (kTilesPerTask * I.tile_vectors - 1 + cvec - 1) / cvec;
  // as many blocks as CUs (one round), each of at least one row
  G.rows_per_block = std::max<uint32_t>(1, (I.rows + (uint32_t)P.cus - 1) / (uint32_t)P.cus);
  G.rows_per_block = std::min<uint32_t>(G.rows_per_block, 16 * kGemmMaxTiles);   // then several rounds
  G.n_blocks = (I.rows + G.rows_per_block - 1) / G.rows_per_block;
  G.groups = std::min<uint32_t>(G.n_blocks, (uint32_t)P.cus);
  G.slab_bytes = (((uint64_t)G.rows_per_block + 2 * G.margin) * I.cols * elem + 255) & ~255ull;
  return EP_OK;
}

uint64_t decode_gemm_workspace(const ep_tensor_info* info, uint32_t elem) {
  GemmGeom G;
  if (!info || gemm_geometry(*info, elem, G)) return 0;
  return kGemmSlabsOffset + (uint64_t)G.groups * G.slab_bytes;
}

// Checks shared by the fused products' entry points.  The INT8 product takes
// the INT8 row container's values (exact int32 sums need C <= 131071); the
// BF16 one takes the bf16 decode of any blob.
int gemm_checks(const ep_tensor_info* info, bool bf, const char* who) {
  if (!info) return fail(EP_ERR_ARG, (std::string(who) + ": null info").c_str());
  if (bf) return EP_OK;
  if (info->container != EP_CONT_INT8_ROW)
    return fail(EP_ERR_UNSUPPORTED, (std::string(who) + ": the tensor is not in the INT8 row container").c_str());
  if (info->cols > 131071)
    return fail(EP_ERR_UNSUPPORTED, (std::string(who) + ": rows longer than 131071 weights may overflow int32").c_str());
  return EP_OK;
}

// Build the tensor's decode tables into the table area at the start of the
// workspace (the same area for both products).
int decode_gemm_prepare(const ep_tensor_info* info, const void* d_blob, void* d_ws, uint64_t ws_bytes,
                        void* stream, bool bf, const char* who) {
  int rc = gemm_checks(info, bf, who);
  if (rc) return rc;
  if (!d_ws || ws_bytes < decode_gemm_workspace(info, bf ? 2 : 1))
    return fail(EP_ERR_ARG, (std::string(who) + ": workspace too small").c_str());
  LayerDev D;
  // the output pointer is never used by the table build
  rc = fill_layer(*info, d_blob, bf ? EP_BF16 : EP_INT8, d_ws, nullptr, 0, info->n_tiles, D, true);
  if (rc) return rc;
  uint8_t* ws = static_cast<uint8_t*>(d_ws);
  D.tables = ws;
  const uint32_t lds = lds_bytes(info->path, *info);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (hipMemcpyAsync(ws + kGemmDescOffset, &D, sizeof D, hipMemcpyHostToDevice, s) != hipSuccess)
    return fail(EP_ERR_HIP, (std::string(who) + ": descriptor copy failed").c_str());
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(&stack_tables_kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return fail(EP_ERR_HIP, (std::string(who) + ": cannot raise the table kernel's LDS limit").c_str());
  hipLaunchKernelGGL(stack_tables_kernel, dim3(1), dim3(kThreads), lds, s,
                     reinterpret_cast<const LayerDev*>(ws + kGemmDescOffset));
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
    return fail(EP_ERR_HIP, (std::string(who) + ": building the decode tables failed").c_str());
  return EP_OK;
}

// The fused decode and MFMA product: INT8 (bf = false: int8 X, int32 Y, the
// INT8 container's values) or BF16 (bf16 X, fp32 Y, the bf16 decode).
// prepared: the workspace holds this tensor's tables (decode_gemm_prepare).
int decode_gemm(const ep_tensor_info* info, const void* d_blob, const void* d_x, int64_t m, void* d_y,
                float* d_dequant, void* d_ws, uint64_t ws_bytes, int32_t* d_status, void* stream,
                bool prepared, bool bf, const char* who) {
  int rc = gemm_checks(info, bf, who);
  if (rc) return rc;
  const std::string w(who);
  const uint32_t elem = bf ? 2 : 1;
  if (m < 1 || m > 65536) return fail(EP_ERR_ARG, (w + ": m must be 1 .. 65536").c_str());
  if (!d_x || !d_y) return fail(EP_ERR_ARG, (w + ": null X or Y").c_str());
  if ((uint64_t)m * info->cols * elem > 0x7FFFFFFFull) return fail(EP_ERR_ARG, (w + ": X above 2^31 bytes").c_str());
  GemmLaunch A;
  std::memset(&A, 0, sizeof A);
  rc = fill_layer(*info, d_blob, bf ? EP_BF16 : EP_INT8, d_y, d_dequant, 0, info->n_tiles, A.L);
  if (rc) return rc;
  GemmGeom G;
  rc = gemm_geometry(*info, elem, G);
  if (rc) return rc;
  if (G.slab_bytes > 0x7FFFFFFFull) return fail(EP_ERR_UNSUPPORTED, (w + ": rows too long").c_str());
  if (!d_ws || ws_bytes < decode_gemm_workspace(info, elem)) return fail(EP_ERR_ARG, (w + ": workspace too small").c_str());
  uint8_t* ws = static_cast<uint8_t*>(d_ws);
  A.L.tables = prepared ? ws : nullptr;
  A.g.x = d_x;
  A.g.y = d_y;
  A.g.slabs = ws + kGemmSlabsOffset;
  A.g.slab_bytes = G.slab_bytes;
  A.g.m = (uint32_t)m;
  A.g.margin = G.margin;
  A.g.n_blocks = G.n_blocks;
  A.g.rows_per_block = G.rows_per_block;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // partial sums are added with atomics (0 is also +0.0f for the BF16 product)
  if (gemm_splits_k((G.rows_per_block + 15) / 16, (uint32_t)((m + 15) / 16)) &&
      !clear_i32(static_cast<int32_t*>(d_y), (int64_t)m * info->rows, s))
    return fail(EP_ERR_HIP, (w + ": clearing Y failed").c_str());
  const uint32_t lds = lds_bytes(info->path, *info);
  DeviceProps P = device_props();
  if (lds > P.max_lds) return fail(EP_ERR_UNSUPPORTED, (w + ": tables exceed the device LDS").c_str());
  const bool wide = gemm_wide((uint32_t)((m + 15) / 16));
  if (set_gemm_lds_limit(info->path, bf, wide, lds) != hipSuccess)
    return fail(EP_ERR_HIP, (w + ": cannot raise the kernel's LDS limit").c_str());
  launch_gemm(info->path, bf, wide, &A, G.groups, lds, d_status, s);
  if (hipGetLastError() != hipSuccess) return fail(EP_ERR_HIP, (w + ": launch failed").c_str());
  return EP_OK;
}

uint64_t decode_layers_workspace(int n) {
  return n > kArgLayers ? (uint64_t)n * sizeof(LayerDev) : 0;
}

// Device descriptors of a layer list, the common decode path, the total task
// count and the LDS bytes of the launch.
int describe_layers(const ep_layer* layers, int n, const char* who, std::vector<LayerDev>& D,
                    uint32_t& path, uint32_t& total, uint32_t& lds) {
  if (n < 0 || (n > 0 && !layers)) return fail(EP_ERR_ARG, (std::string(who) + ": bad layer list").c_str());
  D.assign((size_t)n, LayerDev{});
  path = n ? layers[0].info.path : 0;
  total = 0;
  lds = 0;
  uint64_t tasks = 0;
  for (int i = 0; i < n; i++) {
    const ep_layer& Lr = layers[i];
    if (Lr.info.path != layers[0].info.path) path = kPathMixed;   // one kernel for every family
    int rc = fill_layer(Lr.info, Lr.d_blob, Lr.out_dtype, Lr.d_out, Lr.d_dequant, 0,
                        Lr.info.n_tiles, D[i]);
    if (rc) return rc;
    D[i].task_begin = (uint32_t)tasks;
    tasks += D[i].n_tasks;
    lds = std::max(lds, lds_bytes(Lr.info.path, Lr.info));
  }
  if (tasks > 0xFFFFFFFFull) return fail(EP_ERR_UNSUPPORTED, (std::string(who) + ": too many tiles").c_str());
  total = (uint32_t)tasks;
  use_small_tasks(D, total);
  return EP_OK;
}

int decode_layers(const ep_layer* layers, int n, void* d_ws, uint64_t ws_bytes, int32_t* d_status,
                  void* stream) {
  std::vector<LayerDev> D;
  uint32_t path = 0, total = 0, lds = 0;
  int rc = describe_layers(layers, n, "ep_decode_layers", D, path, total, lds);
  if (rc) return rc;
  if (total == 0) return EP_OK;
  return launch_layers(path, D, total, lds, d_ws, ws_bytes, d_status,
                       static_cast<hipStream_t>(stream), "ep_decode_layers");
}

// ---- decode without any allocation: the descriptor list in a static device array ----
// For callers that cannot allocate device memory.  The descriptors that
// ep_decode_layers copies into the caller's workspace go to `scratch`, a
// file-scope device array that every device running this library holds until
// the process ends.  Host code never names the array as a pointer: its device
// address on each device is looked up once with hipGetSymbolAddress and kept.
constexpr int kNoAllocMaxLayers = 512;
constexpr size_t kScratchBytes = (size_t)kNoAllocMaxLayers * sizeof(LayerDev);
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

// Device address of `scratch` on the current device (looked up on first use
// per device), or an error.
int scratch_address(void** out) {
  static std::mutex mu;
  static std::vector<void*> addr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return fail(EP_ERR_HIP, "ep_decode_layers_noalloc: no HIP device");
  std::lock_guard<std::mutex> g(mu);
  if ((int)addr.size() <= dev) addr.resize((size_t)dev + 1, nullptr);
  if (!addr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
      return fail(EP_ERR_HIP, "ep_decode_layers_noalloc: cannot find the static descriptor array");
    addr[dev] = ptr;
  }
  *out = addr[dev];
  return EP_OK;
}

int decode_layers_noalloc(const ep_layer* layers, int n, int32_t* d_status, void* stream) {
  if (n > kNoAllocMaxLayers)
    return fail(EP_ERR_ARG, "ep_decode_layers_noalloc: more than 512 layers (the static descriptor array's size)");
  std::vector<LayerDev> D;
  uint32_t path = 0, total = 0, lds = 0;
  int rc = describe_layers(layers, n, "ep_decode_layers_noalloc", D, path, total, lds);
  if (rc) return rc;
  if (total == 0) return EP_OK;
  void* ptr = nullptr;
  rc = scratch_address(&ptr);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the previous call's descriptors are simply overwritten (every entry used is written here)
  if (hipMemcpyAsync(ptr, D.data(), sizeof(LayerDev) * D.size(), hipMemcpyHostToDevice, s) != hipSuccess)
    return fail(EP_ERR_HIP, "ep_decode_layers_noalloc: descriptor copy failed");
  return launch_list(path, static_cast<const LayerDev*>(ptr), n, total, lds, d_status, s,
                     "ep_decode_layers_noalloc");
}

// Workspace of a prepared stack: the n descriptors, then one table image per layer
// (every path's tables fit 128 KiB).
uint64_t stack_tables_offset(int n) { return ((uint64_t)n * sizeof(LayerDev) + 255) & ~255ull; }
uint64_t stack_workspace(int n) {
  return n > 0 ? stack_tables_offset(n) + (uint64_t)n * kTableImageBytes : 0;
}

int stack_prepare(const ep_layer* layers, int n, void* d_ws, uint64_t ws_bytes, ep_stack* st,
                  void* stream) {
  if (!st) return fail(EP_ERR_ARG, "ep_stack_prepare: null stack");
  std::memset(st, 0, sizeof *st);
  std::vector<LayerDev> D;
  uint32_t path = 0, total = 0, lds = 0;
  int rc = describe_layers(layers, n, "ep_stack_prepare", D, path, total, lds);
  if (rc) return rc;
  if (n > 0) {
    if (!d_ws || ws_bytes < stack_workspace(n))
      return fail(EP_ERR_ARG, "ep_stack_prepare: workspace too small");
    uint8_t* images = static_cast<uint8_t*>(d_ws) + stack_tables_offset(n);
    uint32_t build_lds = 0;
    for (int i = 0; i < n; i++) {
      D[i].tables = images + (uint64_t)i * kTableImageBytes;
      build_lds = std::max(build_lds, lds_bytes(layers[i].info.path, layers[i].info));
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (hipMemcpyAsync(d_ws, D.data(), sizeof(LayerDev) * D.size(), hipMemcpyHostToDevice, s) != hipSuccess)
      return fail(EP_ERR_HIP, "ep_stack_prepare: descriptor copy failed");
    // the tables are built once here; every ep_stack_decode copies them into LDS
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(&stack_tables_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)build_lds) != hipSuccess)
      return fail(EP_ERR_HIP, "ep_stack_prepare: cannot raise the table kernel's LDS limit");
    hipLaunchKernelGGL(stack_tables_kernel, dim3((unsigned)n), dim3(kThreads), build_lds, s,
                       static_cast<const LayerDev*>(d_ws));
    if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
      return fail(EP_ERR_HIP, "ep_stack_prepare: building the decode tables failed");
  }
  st->d_workspace = d_ws;
  st->n_layers = n;
  st->path = path;
  st->total_tasks = total;
  st->lds_bytes = lds;
  return EP_OK;
}

int stack_decode(const ep_stack* st, int32_t* d_status, void* stream) {
  if (!st || st->n_layers < 0 || (st->n_layers > 0 && !st->d_workspace))
    return fail(EP_ERR_ARG, "ep_stack_decode: stack not prepared");
  if (st->total_tasks == 0) return EP_OK;
  if (!valid_launch_path(st->path)) return fail(EP_ERR_ARG, "ep_stack_decode: stack not prepared");
  return launch_list(st->path, static_cast<const LayerDev*>(st->d_workspace), st->n_layers,
                     st->total_tasks, st->lds_bytes, d_status, static_cast<hipStream_t>(stream),
                     "ep_stack_decode");
}

}  // namespace ep

extern "C" {

int ep_decode_tiles(const ep_tensor_info* info, const void* d_blob, int out_dtype, void* d_out,
                    float* d_dequant, uint32_t tile_begin, uint32_t tile_end, int32_t* d_status,
                    void* hip_stream) {
  return ep::decode_tiles(info, d_blob, out_dtype, d_out, d_dequant, tile_begin, tile_end,
                          d_status, hip_stream);
}

int ep_decode_matmul_i8(const ep_tensor_info* info, const void* d_blob, const int8_t* d_x, int m,
                        int32_t* d_y, float* d_dequant, int32_t* d_status, void* hip_stream) {
  return ep::decode_matmul_i8(info, d_blob, d_x, m, d_y, d_dequant, d_status, hip_stream);
}

uint64_t ep_decode_gemm_i8_workspace(const ep_tensor_info* info) { return ep::decode_gemm_workspace(info, 1); }

int ep_decode_gemm_i8_prepare(const ep_tensor_info* info, const void* d_blob, void* d_workspace,
                              uint64_t ws_bytes, void* hip_stream) {
  return ep::decode_gemm_prepare(info, d_blob, d_workspace, ws_bytes, hip_stream, false,
                                 "ep_decode_gemm_i8_prepare");
}

int ep_decode_gemm_i8_prepared(const ep_tensor_info* info, const void* d_blob, const int8_t* d_x,
                               int64_t m, int32_t* d_y, float* d_dequant, void* d_workspace,
                               uint64_t ws_bytes, int32_t* d_status, void* hip_stream) {
  return ep::decode_gemm(info, d_blob, d_x, m, d_y, d_dequant, d_workspace, ws_bytes, d_status,
                         hip_stream, true, false, "ep_decode_gemm_i8_prepared");
}

int ep_decode_gemm_i8(const ep_tensor_info* info, const void* d_blob, const int8_t* d_x, int64_t m,
                      int32_t* d_y, float* d_dequant, void* d_workspace, uint64_t ws_bytes,
                      int32_t* d_status, void* hip_stream) {
  return ep::decode_gemm(info, d_blob, d_x, m, d_y, d_dequant, d_workspace, ws_bytes, d_status,
                         hip_stream, false, false, "ep_decode_gemm_i8");
}

uint64_t ep_decode_gemm_bf16_workspace(const ep_tensor_info* info) { return ep::decode_gemm_workspace(info, 2); }

int ep_decode_gemm_bf16_prepare(const ep_tensor_info* info, const void* d_blob, void* d_workspace,
                                uint64_t ws_bytes, void* hip_stream) {
  return ep::decode_gemm_prepare(info, d_blob, d_workspace, ws_bytes, hip_stream, true,
                                 "ep_decode_gemm_bf16_prepare");
}

int ep_decode_gemm_bf16(const ep_tensor_info* info, const void* d_blob, const void* d_x, int64_t m,
                        float* d_y, float* d_dequant, void* d_workspace, uint64_t ws_bytes,
                        int32_t* d_status, void* hip_stream) {
  return ep::decode_gemm(info, d_blob, d_x, m, d_y, d_dequant, d_workspace, ws_bytes, d_status,
                         hip_stream, false, true, "ep_decode_gemm_bf16");
}

int ep_decode_gemm_bf16_prepared(const ep_tensor_info* info, const void* d_blob, const void* d_x,
                                 int64_t m, float* d_y, float* d_dequant, void* d_workspace,
                                 uint64_t ws_bytes, int32_t* d_status, void* hip_stream) {
  return ep::decode_gemm(info, d_blob, d_x, m, d_y, d_dequant, d_workspace, ws_bytes, d_status,
                         hip_stream, true, true, "ep_decode_gemm_bf16_prepared");
}

uint64_t ep_decode_layers_workspace(int n) { return ep::decode_layers_workspace(n); }

int ep_decode_layers(const ep_layer* layers, int n, void* d_workspace, uint64_t ws_bytes,
                     int32_t* d_status, void* hip_stream) {
  return ep::decode_layers(layers, n, d_workspace, ws_bytes, d_status, hip_stream);
}

int ep_decode_layers_noalloc(const ep_layer* layers, int n, int32_t* d_status, void* hip_stream) {
  return ep::decode_layers_noalloc(layers, n, d_status, hip_stream);
}

uint64_t ep_stack_workspace(int n) { return ep::stack_workspace(n); }

int ep_stack_prepare(const ep_layer* layers, int n, void* d_workspace, uint64_t ws_bytes,
                     ep_stack* stack, void* hip_stream) {
  return ep::stack_prepare(layers, n, d_workspace, ws_bytes, stack, hip_stream);
}

int ep_stack_decode(const ep_stack* stack, int32_t* d_status, void* hip_stream) {
  return ep::stack_decode(stack, d_status, hip_stream);
}

}  // extern "C"
