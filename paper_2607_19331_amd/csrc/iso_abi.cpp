// extern "C" entry points of libiso.so: argument checks, workspace layout, tensor-table
// upload and kernel sequencing on the caller's stream.  Declarations and the meaning
// of every argument are in include/iso.h.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>
#include <unordered_map>
#include <vector>

#include "iso.h"
#include "iso_device.h"
#include "iso_fused.h"
#include "iso_kernels.h"
#include "iso_ortho.h"
#include "iso_spectral.h"
#include "iso_tsv.h"
#include "iso_update_call.h"

using namespace iso;

namespace {

constexpr int64_t kTieChunk = 1 << 16;
// Per-chunk histograms let the tie search skip a second read of the deltas; above this
// size the library counts ties with an extra pass instead.
constexpr size_t kChunkHistBudget = 16ull << 30;
constexpr int64_t kMaxElems = 0xFFFFFFFFll;   // per tensor: histogram counters are 32-bit

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct Need {
  bool base = false, deltas = false, out = false, k = false;
};

iso_status check_table(const iso_tensor* t, int n_t, int K, int dt, Need need) {
  if (n_t < 0 || (n_t > 0 && t == nullptr)) return ISO_ERR_INVALID_ARG;
  if (K < 1 || K > ISO_MAX_K) return ISO_ERR_INVALID_ARG;
  if (dt != ISO_F32 && dt != ISO_BF16) return ISO_ERR_INVALID_ARG;
  for (int j = 0; j < n_t; ++j) {
    const iso_tensor& x = t[j];
    if (x.rows < 0 || x.cols < 0 || x.select_group < 0) return ISO_ERR_INVALID_ARG;
    if (x.cols != 0 && x.rows > kMaxElems / x.cols) return ISO_ERR_UNSUPPORTED;
    const int64_t n = x.rows * x.cols;
    if (need.k && (x.k < 0 || (x.select_group == 0 && x.k > n))) return ISO_ERR_INVALID_ARG;   // groups: check_groups
    if (n == 0) continue;
    if (need.base) {
      if (!x.base) return ISO_ERR_INVALID_ARG;
      if (!aligned16(x.base)) return ISO_ERR_ALIGNMENT;
    }
    if (need.deltas) {
      for (int i = 0; i < K; ++i) {
        if (!x.deltas[i]) return ISO_ERR_INVALID_ARG;
        if (!aligned16(x.deltas[i])) return ISO_ERR_ALIGNMENT;
      }
    }
    if (need.out) {
      if (!x.out) return ISO_ERR_INVALID_ARG;
      if (!aligned16(x.out)) return ISO_ERR_ALIGNMENT;
    }
  }
  return ISO_OK;
}

iso_status check_ptr_array(const void* const* p, int n, bool required) {
  if (p == nullptr) return required ? ISO_ERR_INVALID_ARG : ISO_OK;
  for (int i = 0; i < n; ++i) {
    if (p[i] == nullptr) return ISO_ERR_INVALID_ARG;
    if (!aligned16(p[i])) return ISO_ERR_ALIGNMENT;
  }
  return ISO_OK;
}

// Joint-selection groups of a table: dense group index per tensor (-1 alone), members of each
// group in table order, the group's count (sum of its members' k) and size.
struct GroupMap {
  int n = 0;
  std::vector<int> gid, mem, mem0;
  std::vector<int64_t> gk, gn;
};

GroupMap group_map(const iso_tensor* t, int n_t) {
  GroupMap G;
  G.gid.assign(n_t, -1);
  std::unordered_map<int32_t, int> index;
  for (int j = 0; j < n_t; ++j) {
    if (t[j].select_group <= 0) continue;
    auto it = index.find(t[j].select_group);
    if (it == index.end()) it = index.emplace(t[j].select_group, (int)index.size()).first;
    G.gid[j] = it->second;
  }
  G.n = (int)index.size();
  G.mem0.assign(G.n + 1, 0);
  G.gk.assign(G.n, 0);
  G.gn.assign(G.n, 0);
  for (int j = 0; j < n_t; ++j)
    if (G.gid[j] >= 0) {
      G.mem0[G.gid[j] + 1] += 1;
      // saturating: a count past any group's size is rejected by check_groups
      const __int128 sum = (__int128)G.gk[G.gid[j]] + t[j].k;
      G.gk[G.gid[j]] = sum > (__int128)INT64_MAX ? INT64_MAX : (int64_t)sum;
      G.gn[G.gid[j]] += t[j].rows * t[j].cols;
    }
  for (int g = 0; g < G.n; ++g) G.mem0[g + 1] += G.mem0[g];
  G.mem.assign(G.mem0[G.n], 0);
  std::vector<int> fill(G.mem0.begin(), G.mem0.end() - 1);
  for (int j = 0; j < n_t; ++j)
    if (G.gid[j] >= 0) G.mem[fill[G.gid[j]]++] = j;
  return G;
}

// Groups are bf16 only, and a group's count cannot exceed its size.  A group may hold more than
// 2^32 entries (its histogram bins are 64-bit); each member stays within the per-tensor limit.
iso_status check_groups(const iso_tensor* t, int n_t, int dt) {
  const GroupMap G = group_map(t, n_t);
  if (G.n == 0) return ISO_OK;
  if (dt != ISO_BF16) return ISO_ERR_UNSUPPORTED;
  for (int g = 0; g < G.n; ++g)
    if (G.gk[g] > G.gn[g]) return ISO_ERR_INVALID_ARG;
  return ISO_OK;
}

// Workspace regions for one call.
struct Layout {
  size_t table = 0, hitem0 = 0, titem0 = 0, ritem0 = 0, ptrs = 0, tmap = 0, upload_end = 0;
  size_t states = 0, hist = 0, tiecnt = 0, desc = 0, chunk_hist = 0;
  size_t fu = 0, tflag = 0, tstat = 0, tinfo = 0, csum = 0, rec = 0;
  size_t spectral = 0;
  size_t ggid = 0, gmem = 0, gmem0 = 0, gk = 0, ghist = 0, gstate = 0, mcnt = 0;
  int n_groups = 0;
  size_t total = 0;
  int64_t hist_chunk = 0, hist_items = 0, tie_items = 0, tiles = 0, groups = 0, ritems = 0, tile_cap = 0;
  bool select = false, use_chunk_hist = false, fused = false;
};

// The single-read TIES path serves bf16 calls that select inside iso_update.
bool fused_eligible(int op, int n_t, int dt) {
  return op == ISO_OP_UPDATE_FUSED_SELECT && dt == ISO_BF16 && n_t <= kFusedMaxTensors;
}

Layout plan(int op, const iso_tensor* t, int n_t, int K, int dt) {
  Layout L;
  size_t off = kStatusBytes;
  L.table = off;
  off = align_up(off + sizeof(DevTensor) * (size_t)n_t, 256);
  L.hitem0 = off;
  off = align_up(off + sizeof(int64_t) * (size_t)n_t, 256);
  L.titem0 = off;
  off = align_up(off + sizeof(int64_t) * (size_t)n_t, 256);
  L.ritem0 = off;
  off = align_up(off + sizeof(int64_t) * (size_t)n_t, 256);
  L.ptrs = off;
  off = align_up(off + sizeof(void*) * (size_t)n_t * K, 256);
  int64_t sumnk = 0;
  for (int j = 0; j < n_t; ++j) sumnk += t[j].rows * t[j].cols * (int64_t)K;
  const int64_t te = merge_tile_elems(dt);
  for (int j = 0; j < n_t; ++j) L.tiles += (t[j].rows * t[j].cols + te - 1) / te;
  L.tmap = off;
  off = align_up(off + sizeof(int) * (size_t)tile_map_entries(L.tiles), 256);
  L.select = (op == ISO_OP_TOPK || op == ISO_OP_UPDATE_FUSED_SELECT);
  if (L.select) {
    const GroupMap G = group_map(t, n_t);
    L.n_groups = G.n;
    if (G.n > 0) {
      L.ggid = off;
      off = align_up(off + sizeof(int) * (size_t)n_t, 256);
      L.gmem = off;
      off = align_up(off + sizeof(int) * (size_t)std::max(1, (int)G.mem.size()), 256);
      L.gmem0 = off;
      off = align_up(off + sizeof(int) * (size_t)(G.n + 1), 256);
      L.gk = off;
      off = align_up(off + sizeof(int64_t) * (size_t)G.n, 256);
    }
  }
  L.upload_end = off;
  if (L.select) {
    L.hist_chunk = hist_chunk_for(sumnk);
    for (int j = 0; j < n_t; ++j) {
      const int64_t n = t[j].rows * t[j].cols;
      L.hist_items += K * ((n + L.hist_chunk - 1) / L.hist_chunk);
      L.tie_items += K * ((n + kTieChunk - 1) / kTieChunk);
    }
    L.states = off;
    off = align_up(off + sizeof(UnitState) * (size_t)n_t * K, 256);
    L.hist = off;
    off = align_up(off + sizeof(uint32_t) * 32768ull * (size_t)n_t * K, 256);
    const size_t ch_bytes = sizeof(uint32_t) * ((size_t)1 << select_last_bits(dt)) * (size_t)L.hist_items;
    L.use_chunk_hist = ch_bytes <= kChunkHistBudget;
    if (L.use_chunk_hist) {
      L.chunk_hist = off;
      off = align_up(off + ch_bytes, 256);
    } else {
      L.tiecnt = off;
      off = align_up(off + sizeof(int32_t) * (size_t)std::max<int64_t>(L.tie_items, 1), 256);
    }
    L.desc = off;
    off = align_up(off + sizeof(iso_select_desc) * (size_t)n_t * K, 256);
    if (L.n_groups > 0) {
      L.ghist = off;
      off = align_up(off + sizeof(uint64_t) * 32768ull * (size_t)L.n_groups * K, 256);
      L.gstate = off;
      off = align_up(off + sizeof(GroupState) * (size_t)L.n_groups * K, 256);
      L.mcnt = off;
      off = align_up(off + sizeof(int64_t) * 2 * (size_t)n_t * K, 256);
    }
  }
  L.fused = fused_eligible(op, n_t, dt) && L.n_groups == 0;
  if (L.fused) {
    for (int j = 0; j < n_t; ++j) L.ritems += fused_reduce_items(t[j].rows * t[j].cols, K);
    for (int j = 0; j < n_t; ++j) L.groups += fused_groups(t[j].rows * t[j].cols);
    L.tile_cap = fused_tile_cap(K);
    const size_t nu = (size_t)n_t * K;
    L.fu = off;
    off = align_up(off + sizeof(FusedUnit) * nu, 256);
    L.tflag = off;
    off = align_up(off + sizeof(int) * (size_t)n_t, 256);
    L.tstat = off;
    off = align_up(off + sizeof(uint16_t) * fused_stat_words(K) * (size_t)L.tiles, 256);
    L.tinfo = off;
    off = align_up(off + sizeof(uint2) * (size_t)L.tiles, 256);
    L.csum = off;
    off = align_up(off + sizeof(uint32_t) * kFusedStat * (size_t)L.ritems, 256);
    L.rec = off;
    off = align_up(off + fused_record_bytes(K) * (size_t)L.tile_cap * (size_t)L.tiles, 256);
  }
  if (op == ISO_OP_UPDATE_SPECTRAL) {
    L.spectral = off;
    off = align_up(off + spectral_workspace_bytes(t, n_t, K), 256);
  }
  if (op == ISO_OP_UPDATE_ORTHO) {
    L.spectral = off;
    off = align_up(off + ortho_workspace_bytes(t, n_t, K), 256);
  }
  L.total = off;
  return L;
}

// Benchmark timing: event pairs recorded around the main streaming kernel of each call.
struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<hipEvent_t> pool;   // 2 per call
  size_t used = 0;
  double flops = 0.0;             // binary64 flops performed inside the timed regions
};
Profiler g_prof;

// Next event pair, or {null, null} when profiling is off (or events cannot be created).
void prof_take(hipEvent_t (&ev)[2]) {
  ev[0] = ev[1] = nullptr;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on) return;
  while (g_prof.pool.size() < g_prof.used + 2) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return;
    g_prof.pool.push_back(e);
  }
  ev[0] = g_prof.pool[g_prof.used];
  ev[1] = g_prof.pool[g_prof.used + 1];
  g_prof.used += 2;
}

struct Upload {
  std::vector<uint8_t> buf;
};
thread_local Upload g_up;   // staging kept alive across calls

// Build [table | hist_item0 | tie_item0 | pointer array] on the host and queue one copy.
hipError_t upload(const Layout& L, const iso_tensor* t, int n_t, int K, int dt, uint8_t* ws,
                  void* const* aux, void* const* aux2, const void* const* ptrs, int n_ptrs, hipStream_t s) {
  g_up.buf.assign(L.upload_end - L.table, 0);
  uint8_t* h = g_up.buf.data();
  DevTensor* tab = (DevTensor*)(h);
  int64_t* hi0 = (int64_t*)(h + (L.hitem0 - L.table));
  int64_t* ti0 = (int64_t*)(h + (L.titem0 - L.table));
  int64_t* ri0 = (int64_t*)(h + (L.ritem0 - L.table));
  const void** pp = (const void**)(h + (L.ptrs - L.table));
  const int64_t te = merge_tile_elems(dt);
  int64_t tile = 0, hitem = 0, titem = 0, ritem = 0, group = 0;
  for (int j = 0; j < n_t; ++j) {
    DevTensor d;
    std::memset(&d, 0, sizeof d);
    d.base = t[j].base;
    for (int i = 0; i < ISO_MAX_K; ++i) d.deltas[i] = (i < K) ? t[j].deltas[i] : nullptr;
    d.out = t[j].out;
    d.aux = aux ? aux[j] : nullptr;
    d.aux2 = aux2 ? aux2[j] : nullptr;
    d.n = t[j].rows * t[j].cols;
    d.k = t[j].k;
    d.tile0 = tile;
    d.group0 = group;
    tab[j] = d;
    tile += (d.n + te - 1) / te;
    group += fused_groups(d.n);
    hi0[j] = hitem;
    ti0[j] = titem;
    ri0[j] = ritem;
    if (L.fused) ritem += fused_reduce_items(d.n, K);
    if (L.select) {
      hitem += K * ((d.n + L.hist_chunk - 1) / L.hist_chunk);
      titem += K * ((d.n + kTieChunk - 1) / kTieChunk);
    }
  }
  for (int q = 0; q < n_ptrs; ++q) pp[q] = ptrs[q];
  if (L.n_groups > 0) {
    const GroupMap G = group_map(t, n_t);
    std::memcpy(h + (L.ggid - L.table), G.gid.data(), sizeof(int) * (size_t)n_t);
    if (!G.mem.empty()) std::memcpy(h + (L.gmem - L.table), G.mem.data(), sizeof(int) * G.mem.size());
    std::memcpy(h + (L.gmem0 - L.table), G.mem0.data(), sizeof(int) * G.mem0.size());
    std::memcpy(h + (L.gk - L.table), G.gk.data(), sizeof(int64_t) * G.gk.size());
  }
  // coarse tile map: the last tensor whose first tile is at or before m << kTileMapShift
  int* tm = (int*)(h + (L.tmap - L.table));
  const int64_t nmap = tile_map_entries(L.tiles);
  for (int64_t m = 0, j = 0; m < nmap; ++m) {
    while (j + 1 < n_t && tab[j + 1].tile0 <= (m << kTileMapShift)) ++j;
    tm[m] = (int)j;
  }
  return hipMemcpyAsync(ws + L.table, h, g_up.buf.size(), hipMemcpyHostToDevice, s);
}

iso_status check_ws(const Layout& L, void* ws, size_t ws_bytes) {
  if (ws == nullptr) return ISO_ERR_WORKSPACE;
  if (((uintptr_t)ws & 255u) != 0) return ISO_ERR_ALIGNMENT;
  if (ws_bytes < L.total) return ISO_ERR_WORKSPACE;
  return ISO_OK;
}

// The workspace of a call once its layout is known: the caller's, checked, or one handed out by
// src.acquire (which rejects a layout it cannot hold).
iso_status take_ws(const WsSource& src, const Layout& L, uint8_t** w) {
  void* ws = src.ws;
  size_t bytes = src.bytes;
  if (src.acquire != nullptr) {
    const iso_status st = src.acquire(L.total, &ws, &bytes);
    if (st != ISO_OK) return st;
  }
  const iso_status st = check_ws(L, ws, bytes);
  if (st == ISO_OK) *w = (uint8_t*)ws;
  return st;
}

#define HIP_TRY(x)                               \
  do {                                           \
    if ((x) != hipSuccess) return ISO_ERR_HIP;   \
  } while (0)

SelectPlan select_plan(const Layout& L, uint8_t* ws, int n_t, int K, iso_select_desc* desc) {
  SelectPlan p;
  p.tab = (const DevTensor*)(ws + L.table);
  p.n_t = n_t;
  p.K = K;
  p.states = (UnitState*)(ws + L.states);
  p.hist = (uint32_t*)(ws + L.hist);
  p.hist_item0 = (const int64_t*)(ws + L.hitem0);
  p.hist_chunk = L.hist_chunk;
  p.hist_items = L.hist_items;
  p.tie_item0 = (const int64_t*)(ws + L.titem0);
  p.tie_chunk = kTieChunk;
  p.tie_items = L.tie_items;
  p.tie_cnt = L.use_chunk_hist ? nullptr : (int32_t*)(ws + L.tiecnt);
  p.chunk_hist = L.use_chunk_hist ? (uint32_t*)(ws + L.chunk_hist) : nullptr;
  p.desc = desc;
  p.status = (uint32_t*)ws;
  if (L.n_groups > 0) {
    p.n_groups = L.n_groups;
    p.gid = (const int*)(ws + L.ggid);
    p.gmem = (const int*)(ws + L.gmem);
    p.gmem0 = (const int*)(ws + L.gmem0);
    p.gk = (const int64_t*)(ws + L.gk);
    p.ghist = (uint64_t*)(ws + L.ghist);
    p.gstate = (GroupState*)(ws + L.gstate);
    p.mcnt = (int64_t*)(ws + L.mcnt);
  }
  return p;
}

hipError_t start_call(uint8_t* ws, hipStream_t s) { return fill_u32((uint32_t*)ws, kStatusBytes / 4, 0u, s); }

hipError_t do_select(const Layout& L, uint8_t* ws, int n_t, int K, int dt, iso_select_desc* desc,
                     hipStream_t s) {
  hipError_t e = fill_u32((uint32_t*)(ws + L.hist), 32768ll * n_t * K, 0u, s);
  if (e != hipSuccess) return e;
  return run_select(select_plan(L, ws, n_t, K, desc), dt, s);
}

int64_t max_numel(const iso_tensor* t, int n_t) {
  int64_t m = 0;
  for (int j = 0; j < n_t; ++j) m = std::max(m, t[j].rows * t[j].cols);
  return m;
}

}  // namespace

extern "C" {

size_t iso_workspace_size(int op, const iso_tensor* t, int n_t, int K, int dt) {
  if (n_t < 0 || (n_t > 0 && !t) || K < 1 || K > ISO_MAX_K) return 0;
  if (op < ISO_OP_TOPK || op > ISO_OP_UPDATE_ORTHO) return 0;
  for (int j = 0; j < n_t; ++j)
    if (t[j].rows < 0 || t[j].cols < 0) return 0;
  if (op == ISO_OP_BLOCKDIAG) return 0;
  return plan(op, t, n_t, K, dt).total;
}

iso_status iso_topk_mask(const iso_tensor* t, int n_t, int K, int dt, iso_select_desc* desc,
                         uint32_t* const* mask_bits, void* ws, size_t ws_bytes, void* stream) {
  Need nd;
  nd.deltas = true;
  nd.k = true;
  iso_status st = check_table(t, n_t, K, dt, nd);
  if (st != ISO_OK) return st;
  if ((st = check_groups(t, n_t, dt)) != ISO_OK) return st;
  if (n_t == 0) return ISO_OK;
  if (desc == nullptr) return ISO_ERR_INVALID_ARG;
  if (((uintptr_t)desc & 7u) != 0) return ISO_ERR_ALIGNMENT;
  if (mask_bits != nullptr)
    for (int q = 0; q < n_t * K; ++q)
      if (mask_bits[q] == nullptr || ((uintptr_t)mask_bits[q] & 3u) != 0) return ISO_ERR_INVALID_ARG;
  Layout L = plan(ISO_OP_TOPK, t, n_t, K, dt);
  if ((st = check_ws(L, ws, ws_bytes)) != ISO_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = (uint8_t*)ws;
  HIP_TRY(start_call(w, s));
  HIP_TRY(upload(L, t, n_t, K, dt, w, nullptr, nullptr, (const void* const*)mask_bits, mask_bits ? n_t * K : 0, s));
  HIP_TRY(do_select(L, w, n_t, K, dt, desc, s));
  if (mask_bits != nullptr)
    HIP_TRY(run_mask_bits((const DevTensor*)(w + L.table), n_t, K, dt, desc, (uint32_t* const*)(w + L.ptrs),
                          max_numel(t, n_t), s));
  return ISO_OK;
}

iso_status iso_sign_elect(const iso_tensor* t, int n_t, int K, int dt, const iso_select_desc* desc,
                          int8_t* const* sign_out, void* ws, size_t ws_bytes, void* stream) {
  Need nd;
  nd.deltas = true;
  iso_status st = check_table(t, n_t, K, dt, nd);
  if (st != ISO_OK) return st;
  if (n_t == 0) return ISO_OK;
  if ((st = check_ptr_array((const void* const*)sign_out, n_t, true)) != ISO_OK) return st;
  Layout L = plan(ISO_OP_SIGN, t, n_t, K, dt);
  if ((st = check_ws(L, ws, ws_bytes)) != ISO_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = (uint8_t*)ws;
  HIP_TRY(start_call(w, s));
  HIP_TRY(upload(L, t, n_t, K, dt, w, (void* const*)sign_out, nullptr, nullptr, 0, s));
  MergePlan mp;
  mp.tab = (const DevTensor*)(w + L.table);
  mp.n_t = n_t;
  mp.K = K;
  mp.mode = ISO_MERGE_TIES;
  mp.outs = OUT_SIGN;
  mp.desc = desc;
  mp.lambda = 1.0;
  mp.eps = 0.0;
  mp.tiles = L.tiles;
  mp.status = (uint32_t*)w;
  HIP_TRY(run_merge(mp, dt, s));
  return ISO_OK;
}

iso_status iso_merge(const iso_tensor* t, int n_t, int K, int dt, int mode,
                     const iso_select_desc* desc, double lambda, double eps_act, float* const* tau_out, void* ws,
                     size_t ws_bytes, void* stream) {
  Need nd;
  nd.deltas = true;
  iso_status st = check_table(t, n_t, K, dt, nd);
  if (st != ISO_OK) return st;
  if (mode != ISO_MERGE_TA && mode != ISO_MERGE_TIES && mode != ISO_MERGE_RAM) return ISO_ERR_INVALID_ARG;
  if (!(lambda == lambda) || !(eps_act == eps_act) || !(eps_act >= 0)) return ISO_ERR_INVALID_ARG;
  if (n_t == 0) return ISO_OK;
  if (mode == ISO_MERGE_TIES && desc == nullptr) return ISO_ERR_INVALID_ARG;
  if ((st = check_ptr_array((const void* const*)tau_out, n_t, true)) != ISO_OK) return st;
  Layout L = plan(ISO_OP_MERGE, t, n_t, K, dt);
  if ((st = check_ws(L, ws, ws_bytes)) != ISO_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = (uint8_t*)ws;
  HIP_TRY(start_call(w, s));
  HIP_TRY(upload(L, t, n_t, K, dt, w, (void* const*)tau_out, nullptr, nullptr, 0, s));
  MergePlan mp;
  mp.tab = (const DevTensor*)(w + L.table);
  mp.n_t = n_t;
  mp.K = K;
  mp.mode = mode;
  mp.outs = OUT_TAU;
  mp.desc = (mode == ISO_MERGE_TIES) ? desc : nullptr;
  mp.lambda = lambda;
  mp.eps = eps_act;
  mp.tiles = L.tiles;
  mp.status = (uint32_t*)w;
  HIP_TRY(run_merge(mp, dt, s));
  return ISO_OK;
}

iso_status iso_update(const iso_tensor* t, int n_t, int K, int dt, const iso_update_args* a, void* ws,
                      size_t ws_bytes, void* stream) {
  WsSource src;
  src.ws = ws;
  src.bytes = ws_bytes;
  return update_call(t, n_t, K, dt, a, src, stream);
}

}  // extern "C"

namespace iso {

void profile_region(hipEvent_t (&ev)[2]) { prof_take(ev); }

void profile_add_flops(double flops) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (g_prof.on) g_prof.flops += flops;
}

// The body of iso_update.  Arguments are validated first; the workspace is then taken from src
// (the caller's, or the fixed per-device block of iso_update_noalloc) once its size is known.
iso_status update_call(const iso_tensor* t, int n_t, int K, int dt, const iso_update_args* a,
                       const WsSource& src, void* stream) {
  if (a == nullptr) return ISO_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = nullptr;
  iso_status st;
  if (a->mode == ISO_UPDATE_APPLY) {
    Need nd;
    nd.base = nd.out = true;
    if ((st = check_table(t, n_t, 1, dt, nd)) != ISO_OK) return st;
    if (!(a->lambda == a->lambda)) return ISO_ERR_INVALID_ARG;
    if (n_t == 0) return ISO_OK;
    if ((st = check_ptr_array((const void* const*)a->tau_in, n_t, true)) != ISO_OK) return st;
    Layout L = plan(ISO_OP_UPDATE_APPLY, t, n_t, 1, dt);
    if ((st = take_ws(src, L, &w)) != ISO_OK) return st;
    HIP_TRY(start_call(w, s));
    HIP_TRY(upload(L, t, n_t, 1, dt, w, (void* const*)a->tau_in, nullptr, nullptr, 0, s));
    HIP_TRY(run_apply((const DevTensor*)(w + L.table), n_t, dt, a->lambda, L.tiles, (uint32_t*)w, s));
    return ISO_OK;
  }
  if (a->mode == ISO_UPDATE_FUSED) {
    const bool ties = a->merge == ISO_MERGE_TIES;
    if (a->merge != ISO_MERGE_TA && !ties && a->merge != ISO_MERGE_RAM) return ISO_ERR_INVALID_ARG;
    Need nd;
    nd.base = nd.out = nd.deltas = true;
    nd.k = ties && a->desc == nullptr;
    if ((st = check_table(t, n_t, K, dt, nd)) != ISO_OK) return st;
    if (nd.k && (st = check_groups(t, n_t, dt)) != ISO_OK) return st;
    if (!(a->lambda == a->lambda) || !(a->eps_act == a->eps_act) || !(a->eps_act >= 0)) return ISO_ERR_INVALID_ARG;
    if (n_t == 0) return ISO_OK;
    const bool want_sign = ties && a->sign_out != nullptr;
    if (want_sign && (st = check_ptr_array((const void* const*)a->sign_out, n_t, true)) != ISO_OK) return st;
    const bool inner_select = ties && a->desc == nullptr;
    Layout L = plan(inner_select ? ISO_OP_UPDATE_FUSED_SELECT : ISO_OP_UPDATE_FUSED, t, n_t, K, dt);
    if ((st = take_ws(src, L, &w)) != ISO_OK) return st;
    HIP_TRY(start_call(w, s));
    HIP_TRY(upload(L, t, n_t, K, dt, w, nullptr, want_sign ? (void* const*)a->sign_out : nullptr, nullptr, 0, s));
    MergePlan mp;
    mp.tab = (const DevTensor*)(w + L.table);
    mp.n_t = n_t;
    mp.K = K;
    mp.mode = a->merge;
    mp.outs = OUT_W | (want_sign ? OUT_SIGN : 0);
    mp.desc = ties ? a->desc : nullptr;
    mp.lambda = a->lambda;
    mp.eps = a->eps_act;
    mp.tiles = L.tiles;
    mp.status = (uint32_t*)w;
    if (L.fused) {
      iso_select_desc* dd = (iso_select_desc*)(w + L.desc);
      FusedPlan fp;
      fp.tab = mp.tab;
      fp.tmap = (const int*)(w + L.tmap);
      fp.n_t = n_t;
      fp.K = K;
      fp.tiles = L.tiles;
      fp.groups = L.groups;
      fp.fu = (FusedUnit*)(w + L.fu);
      fp.tflag = (int*)(w + L.tflag);
      fp.tstat = (uint16_t*)(w + L.tstat);
      fp.tinfo = (uint2*)(w + L.tinfo);
      fp.rec = (uint32_t*)(w + L.rec);
      fp.tile_cap = L.tile_cap;
      fp.ritem0 = (const int64_t*)(w + L.ritem0);
      fp.ritems = L.ritems;
      fp.csum = (uint32_t*)(w + L.csum);
      fp.lambda = a->lambda;
      fp.want_sign = want_sign ? 1 : 0;
      fp.status = (uint32_t*)w;
      fp.sel = select_plan(L, w, n_t, K, dd);
      fp.mrg = mp;
      if (!src.acquire) prof_take(fp.prof);
      HIP_TRY(run_fused(fp, s));
      return ISO_OK;
    }
    if (inner_select) {
      iso_select_desc* dd = (iso_select_desc*)(w + L.desc);
      HIP_TRY(do_select(L, w, n_t, K, dt, dd, s));
      mp.desc = dd;
    }
    if (!src.acquire) prof_take(mp.prof);
    HIP_TRY(run_merge(mp, dt, s));
    return ISO_OK;
  }
  if (a->mode == ISO_UPDATE_SPECTRAL) {
    Need nd;
    nd.base = nd.out = nd.deltas = true;
    if ((st = check_table(t, n_t, K, dt, nd)) != ISO_OK) return st;
    if (!(a->rho_keep > 0.0 && a->rho_keep <= 1.0) || !(a->ridge >= 0.0) || !(a->c_min <= a->c_max))
      return ISO_ERR_INVALID_ARG;
    for (int j = 0; j < n_t; ++j)
      if (std::min(t[j].rows, t[j].cols) > ISO_SPECTRAL_MAX_DIM) return ISO_ERR_UNSUPPORTED;
    if (a->coef_out != nullptr && ((uintptr_t)a->coef_out & 7u) != 0) return ISO_ERR_ALIGNMENT;
    if (n_t == 0) return ISO_OK;
    Layout L = plan(ISO_OP_UPDATE_SPECTRAL, t, n_t, K, dt);
    if ((st = take_ws(src, L, &w)) != ISO_OK) return st;
    HIP_TRY(start_call(w, s));
    SpectralArgs sa;
    sa.rho_keep = a->rho_keep;
    sa.ridge = a->ridge;
    sa.c_min = a->c_min;
    sa.c_max = a->c_max;
    sa.coef_out = a->coef_out;
    return run_spectral(t, n_t, K, (iso_dtype)dt, sa, w + L.spectral, (uint32_t*)w, s);
  }
  if (a->mode == ISO_UPDATE_ORTHO) {
    Need nd;
    nd.base = nd.out = nd.deltas = nd.k = true;
    if ((st = check_table(t, n_t, K, dt, nd)) != ISO_OK) return st;
    if (!(a->lambda - a->lambda == 0.0)) return ISO_ERR_INVALID_ARG;
    for (int j = 0; j < n_t; ++j) {
      if (t[j].select_group != 0) return ISO_ERR_UNSUPPORTED;
      if (t[j].rows * t[j].cols == 0) continue;
      if (t[j].rows < t[j].cols || t[j].cols > ISO_SPECTRAL_MAX_DIM) return ISO_ERR_UNSUPPORTED;
    }
    if (n_t == 0) return ISO_OK;
    Layout L = plan(ISO_OP_UPDATE_ORTHO, t, n_t, K, dt);
    if ((st = take_ws(src, L, &w)) != ISO_OK) return st;
    HIP_TRY(start_call(w, s));
    return run_ortho(t, n_t, K, (iso_dtype)dt, a->lambda, w + L.spectral, (uint32_t*)w, s);
  }
  return ISO_ERR_INVALID_ARG;
}

}  // namespace iso

extern "C" {

static iso_status check_tsv(const iso_tensor* t, int n_t, int K, int dt, int rank, bool ptrs) {
  Need nd;
  nd.base = nd.out = nd.deltas = ptrs;
  iso_status st = check_table(t, n_t, K, dt, nd);
  if (st != ISO_OK) return st;
  if (rank < 1) return ISO_ERR_INVALID_ARG;
  if (dt != ISO_BF16) return ISO_ERR_UNSUPPORTED;
  int width = -1;
  for (int j = 0; j < n_t; ++j) {
    const int64_t q = std::min(t[j].rows, t[j].cols);
    if ((int64_t)K * rank > q) return ISO_ERR_INVALID_ARG;
    const int L = tsv_sketch_width(t[j].rows, t[j].cols, rank);
    if (L == 0) return ISO_ERR_UNSUPPORTED;
    if (width >= 0 && L != width) return ISO_ERR_UNSUPPORTED;   // one sketch width per call
    width = L;
  }
  return ISO_OK;
}

size_t iso_workspace_size_tsv(const iso_tensor* t, int n_t, int K, int dt, int rank) {
  if (check_tsv(t, n_t, K, dt, rank, false) != ISO_OK) return 0;
  return kStatusBytes + tsv_workspace_bytes(t, n_t, K, rank);
}

iso_status iso_blockdiag_project(const iso_tensor* t, int n_t, int K, int dt, int rank, double alpha,
                                 float* const* delta_hat, void* ws, size_t ws_bytes, void* stream) {
  iso_status st = check_tsv(t, n_t, K, dt, rank, true);
  if (st != ISO_OK) return st;
  if (!(alpha - alpha == 0.0)) return ISO_ERR_INVALID_ARG;
  if (n_t == 0) return ISO_OK;
  if (delta_hat != nullptr && (st = check_ptr_array((const void* const*)delta_hat, n_t, true)) != ISO_OK) return st;
  const size_t need = kStatusBytes + tsv_workspace_bytes(t, n_t, K, rank);
  if (ws == nullptr) return ISO_ERR_WORKSPACE;
  if (((uintptr_t)ws & 255u) != 0) return ISO_ERR_ALIGNMENT;
  if (ws_bytes < need) return ISO_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = (uint8_t*)ws;
  HIP_TRY(start_call(w, s));
  TsvArgs ta;
  ta.rank = rank;
  ta.alpha = alpha;
  ta.delta_hat = delta_hat;
  return run_tsv(t, n_t, K, ta, w + kStatusBytes, ws_bytes - kStatusBytes, (uint32_t*)w, s);
}

iso_status iso_blockdiag_project_factors(const iso_tensor* t, int n_t, int K, int dt, int rank, double alpha,
                                         const iso_factors* factors, float* const* delta_hat, void* ws,
                                         size_t ws_bytes, void* stream) {
  iso_status st = check_tsv(t, n_t, K, dt, rank, false);
  if (st != ISO_OK) return st;
  Need nd;
  nd.base = nd.out = true;
  if ((st = check_table(t, n_t, K, dt, nd)) != ISO_OK) return st;
  if (!(alpha - alpha == 0.0)) return ISO_ERR_INVALID_ARG;
  if (n_t == 0) return ISO_OK;
  if (factors == nullptr) return ISO_ERR_INVALID_ARG;
  for (int q = 0; q < n_t * K; ++q)
    if (factors[q].u == nullptr || factors[q].s == nullptr || factors[q].v == nullptr) return ISO_ERR_INVALID_ARG;
  if (delta_hat != nullptr && (st = check_ptr_array((const void* const*)delta_hat, n_t, true)) != ISO_OK) return st;
  const size_t need = kStatusBytes + tsv_workspace_bytes(t, n_t, K, rank);
  if (ws == nullptr) return ISO_ERR_WORKSPACE;
  if (((uintptr_t)ws & 255u) != 0) return ISO_ERR_ALIGNMENT;
  if (ws_bytes < need) return ISO_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = (uint8_t*)ws;
  HIP_TRY(start_call(w, s));
  TsvArgs ta;
  ta.rank = rank;
  ta.alpha = alpha;
  ta.delta_hat = delta_hat;
  ta.factors = factors;
  return run_tsv(t, n_t, K, ta, w + kStatusBytes, ws_bytes - kStatusBytes, (uint32_t*)w, s);
}

static iso_status spectrum_op(const iso_tensor* t, int n_t, int dt, SpectrumOp op, double* out, double param,
                              void* ws, size_t ws_bytes, void* stream, const double* fracs = nullptr, int n_frac = 0) {
  const bool write = op == SpectrumOp::kInterpolate;
  Need nd;
  nd.base = true;
  nd.deltas = op != SpectrumOp::kSelfSpectralError;
  nd.out = write;
  iso_status st = check_table(t, n_t, 1, dt, nd);
  if (st != ISO_OK) return st;
  for (int j = 0; j < n_t; ++j)
    if (std::min(t[j].rows, t[j].cols) > ISO_SPECTRAL_MAX_DIM) return ISO_ERR_UNSUPPORTED;
  if (!write && (out == nullptr || ((uintptr_t)out & 7u) != 0)) return out ? ISO_ERR_ALIGNMENT : ISO_ERR_INVALID_ARG;
  if (write && !(param - param == 0.0)) return ISO_ERR_INVALID_ARG;
  if (op == SpectrumOp::kTransport) {
    if (fracs == nullptr || n_frac < 1 || n_frac > ISO_MAX_RANK_FRACS) return ISO_ERR_INVALID_ARG;
    for (int i = 0; i < n_frac; ++i)
      if (!(fracs[i] > 0.0 && fracs[i] <= 1.0)) return ISO_ERR_INVALID_ARG;
  }
  if (n_t == 0) return ISO_OK;
  Layout L = plan(ISO_OP_UPDATE_SPECTRAL, t, n_t, 1, dt);
  if ((st = check_ws(L, ws, ws_bytes)) != ISO_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = (uint8_t*)ws;
  HIP_TRY(start_call(w, s));
  return run_spectrum_ops(t, n_t, (iso_dtype)dt, op, out, param, fracs, n_frac, w + L.spectral, (uint32_t*)w, s);
}

// second_moments: the AdamW state v_u, v_v must be given (Muon does not use them).
static iso_status check_frames(const iso_frame* f, int n_f, bool second_moments = true) {
  if (n_f < 0 || (n_f > 0 && f == nullptr)) return ISO_ERR_INVALID_ARG;
  for (int e = 0; e < n_f; ++e) {
    const iso_frame& F = f[e];
    if (F.rows < 1 || F.cols < 1 || F.rank < 1 || F.rank > std::min(F.rows, F.cols)) return ISO_ERR_INVALID_ARG;
    if (std::min(F.rows, F.cols) > ISO_SPECTRAL_MAX_DIM || std::max(F.rows, F.cols) > kMaxElems / std::min(F.rows, F.cols))
      return ISO_ERR_UNSUPPORTED;
    const void* p[9] = {F.u, F.v, F.sigma, F.m_u, F.v_u, F.m_v, F.v_v, F.grad, F.w_out};
    for (int q = 0; q < 9; ++q) {
      const bool used = second_moments || (q != 4 && q != 6);
      if (used && p[q] == nullptr) return ISO_ERR_INVALID_ARG;
    }
    for (int q = 0; q < 7; ++q)
      if (((uintptr_t)p[q] & 7u) != 0) return ISO_ERR_ALIGNMENT;
    if (((uintptr_t)F.grad & 3u) != 0 || ((uintptr_t)F.w_out & 3u) != 0) return ISO_ERR_ALIGNMENT;
  }
  return ISO_OK;
}

size_t iso_workspace_size_optimizer(const iso_frame* f, int n_f) {
  if (check_frames(f, n_f, false) != ISO_OK) return 0;
  return kStatusBytes + optimizer_workspace_bytes(f, n_f);
}

iso_status iso_optimizer_step(const iso_frame* f, int n_f, int dt, const iso_adamw* opt, void* ws,
                              size_t ws_bytes, void* stream) {
  iso_status st = check_frames(f, n_f);
  if (st != ISO_OK) return st;
  if (dt != ISO_F32 && dt != ISO_BF16) return ISO_ERR_INVALID_ARG;
  if (opt == nullptr || opt->step < 1) return ISO_ERR_INVALID_ARG;
  const double h[5] = {opt->lr, opt->beta1, opt->beta2, opt->eps, opt->weight_decay};
  for (double x : h)
    if (!(x - x == 0.0)) return ISO_ERR_INVALID_ARG;
  if (!(opt->beta1 >= 0.0 && opt->beta1 < 1.0 && opt->beta2 >= 0.0 && opt->beta2 < 1.0 && opt->eps > 0.0))
    return ISO_ERR_INVALID_ARG;
  if (n_f == 0) return ISO_OK;
  const size_t need = kStatusBytes + optimizer_workspace_bytes(f, n_f);
  if (ws == nullptr) return ISO_ERR_WORKSPACE;
  if (((uintptr_t)ws & 255u) != 0) return ISO_ERR_ALIGNMENT;
  if (ws_bytes < need) return ISO_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = (uint8_t*)ws;
  HIP_TRY(start_call(w, s));
  return run_optimizer(f, n_f, (iso_dtype)dt, opt, nullptr, w + kStatusBytes, (uint32_t*)w, s);
}

iso_status iso_optimizer_step_muon(const iso_frame* f, int n_f, int dt, const iso_muon* opt, void* ws,
                                   size_t ws_bytes, void* stream) {
  iso_status st = check_frames(f, n_f, false);
  if (st != ISO_OK) return st;
  if (dt != ISO_F32 && dt != ISO_BF16) return ISO_ERR_INVALID_ARG;
  if (opt == nullptr) return ISO_ERR_INVALID_ARG;
  const double h[3] = {opt->lr, opt->momentum, opt->weight_decay};
  for (double x : h)
    if (!(x - x == 0.0)) return ISO_ERR_INVALID_ARG;
  if (!(opt->momentum >= 0.0 && opt->momentum < 1.0)) return ISO_ERR_INVALID_ARG;
  if (n_f == 0) return ISO_OK;
  const size_t need = kStatusBytes + optimizer_workspace_bytes(f, n_f);
  if (ws == nullptr) return ISO_ERR_WORKSPACE;
  if (((uintptr_t)ws & 255u) != 0) return ISO_ERR_ALIGNMENT;
  if (ws_bytes < need) return ISO_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* w = (uint8_t*)ws;
  HIP_TRY(start_call(w, s));
  return run_optimizer(f, n_f, (iso_dtype)dt, nullptr, opt, w + kStatusBytes, (uint32_t*)w, s);
}

iso_status iso_spectral_diagnostics(const iso_tensor* t, int n_t, int dt, double* out, void* ws,
                                    size_t ws_bytes, void* stream) {
  return spectrum_op(t, n_t, dt, SpectrumOp::kDiagnostics, out, 0.0, ws, ws_bytes, stream);
}

iso_status iso_spectral_error(const iso_tensor* t, int n_t, int dt, int self_recon, double* out, void* ws,
                              size_t ws_bytes, void* stream) {
  if (self_recon != 0 && self_recon != 1) return ISO_ERR_INVALID_ARG;
  return spectrum_op(t, n_t, dt, self_recon ? SpectrumOp::kSelfSpectralError : SpectrumOp::kSpectralError, out, 0.0,
                     ws, ws_bytes, stream);
}

iso_status iso_spectrum_interpolate(const iso_tensor* t, int n_t, int dt, double alpha, void* ws,
                                    size_t ws_bytes, void* stream) {
  return spectrum_op(t, n_t, dt, SpectrumOp::kInterpolate, nullptr, alpha, ws, ws_bytes, stream);
}

iso_status iso_transport_ratios(const iso_tensor* t, int n_t, int dt, const double* rank_frac, int n_frac,
                                double* out, void* ws, size_t ws_bytes, void* stream) {
  return spectrum_op(t, n_t, dt, SpectrumOp::kTransport, out, 0.0, ws, ws_bytes, stream, rank_frac, n_frac);
}

int64_t iso_k_from_density(int64_t n, int64_t num, int64_t den) {
  if (n < 0 || num < 0 || den <= 0 || num > den) return -1;
  __int128 v = (__int128)2 * n * num + den;
  return (int64_t)(v / ((__int128)2 * den));
}

iso_status iso_read_device_status(const void* ws, void* stream) {
  if (ws == nullptr) return ISO_ERR_INVALID_ARG;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return ISO_ERR_HIP;
  uint32_t flags = 0;
  if (hipMemcpy(&flags, ws, sizeof flags, hipMemcpyDeviceToHost) != hipSuccess) return ISO_ERR_HIP;
  if (flags & kStatusInternal) return ISO_ERR_INTERNAL;
  if (flags & kStatusNonFinite) return ISO_ERR_NONFINITE;
  return ISO_OK;
}

iso_status iso_profile_begin(void) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = true;
  g_prof.used = 0;
  g_prof.flops = 0.0;
  return ISO_OK;
}

iso_status iso_profile_flops(double* flops) {
  if (flops == nullptr) return ISO_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  *flops = g_prof.flops;
  return ISO_OK;
}

iso_status iso_profile_end(double* total_ms, int32_t* launches) {
  if (total_ms == nullptr || launches == nullptr) return ISO_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = false;
  double sum = 0.0;
  for (size_t q = 0; q + 1 < g_prof.used; q += 2) {
    if (hipEventSynchronize(g_prof.pool[q + 1]) != hipSuccess) return ISO_ERR_HIP;
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, g_prof.pool[q], g_prof.pool[q + 1]) != hipSuccess) return ISO_ERR_HIP;
    sum += ms;
  }
  *total_ms = sum;
  *launches = (int32_t)(g_prof.used / 2);
  g_prof.used = 0;
  return ISO_OK;
}

iso_status iso_read_fallback_count(const void* ws, void* stream, int32_t* count) {
  if (ws == nullptr || count == nullptr) return ISO_ERR_INVALID_ARG;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return ISO_ERR_HIP;
  uint32_t v = 0;
  if (hipMemcpy(&v, (const uint32_t*)ws + 1, sizeof v, hipMemcpyDeviceToHost) != hipSuccess) return ISO_ERR_HIP;
  *count = (int32_t)v;
  return ISO_OK;
}

const char* iso_status_string(int s) {
  switch (s) {
    case ISO_OK: return "ok";
    case ISO_ERR_INVALID_ARG: return "invalid argument";
    case ISO_ERR_ALIGNMENT: return "pointer not 16-byte aligned";
    case ISO_ERR_WORKSPACE: return "workspace missing or too small";
    case ISO_ERR_NONFINITE: return "non-finite input value";
    case ISO_ERR_HIP: return "HIP runtime error";
    case ISO_ERR_UNSUPPORTED: return "unsupported shape or option";
    case ISO_ERR_INTERNAL: return "internal consistency check failed";
  }
  return "unknown status";
}

}  // extern "C"
