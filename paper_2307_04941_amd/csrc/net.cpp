// Network executor: chains of convolution and max-pooling layers run back to
// back on one device (the convolution stacks of the networks of Sec. 5.2).
//
// At creation every activation's shape is inferred and every convolution
// planned once; activations are packed into one device arena by liveness
// (an activation's space is reused once no later layer reads it) and the
// split-K partials of all convolutions share one workspace, since the layers
// run in order on one stream.  A forward pass is then only kernel launches;
// mg3m_net_forward_graph captures those launches into a HIP graph once and
// replays it, which removes the per-launch host cost for networks of many
// small layers.
//
// Every layer runs in HWCN, the tuned layout, whatever the network's layout.
// An NCHW network changes layout only at its edges: its input is copied to
// HWCN in the arena, its filters to [R][S][C][K] in a buffer of the network's
// own, and its last layer's HWCN output to the caller's NCHW y, each by one
// kernel per forward pass.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <exception>
#include <string>
#include <vector>

#include "mg3m.h"
#include "mg3m_internal.h"

struct mg3m_net {
  int layout = 0, N = 0, device = 0;   // layout: of x, y and the filters; the layers run in HWCN
  std::vector<mg3m_layer> layers;
  std::vector<int> C, H, W;            // per activation 0 .. n
  std::vector<long long> offset;       // byte offset in the arena; -1 for the input and the output
  char* arena = nullptr;
  size_t arena_bytes = 0;
  void* ws = nullptr;
  size_t ws_bytes = 0;
  // NCHW networks: HWCN filter copies, one block per convolution (offset per layer, -1 for pooling)
  float* wt = nullptr;
  size_t wt_bytes = 0;
  std::vector<long long> wt_off;
  // ... and the layout changes that make them, one batch per forward pass
  // (the job table in device memory)
  mg3m::SwapJob* wt_jobs = nullptr;
  int wt_njobs = 0;
  unsigned wt_tiles = 0;
  // captured forward pass
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  const float* gx = nullptr;
  float* gy = nullptr;
  hipStream_t gs = nullptr;
};

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

std::string at(int i) { return "layer " + std::to_string(i) + ": "; }

// First-fit packing of activation buffers into one arena.  Blocks are kept
// sorted by offset; a freed block is merged with free neighbours.
struct Arena {
  struct Block { size_t off, size; bool used; };
  std::vector<Block> blocks;
  size_t end = 0;

  size_t take(size_t size) {
    for (size_t i = 0; i < blocks.size(); ++i) {
      Block& b = blocks[i];
      if (b.used || b.size < size) continue;
      if (b.size > size) blocks.insert(blocks.begin() + i + 1, Block{b.off + size, b.size - size, false});
      blocks[i].size = size;
      blocks[i].used = true;
      return blocks[i].off;
    }
    if (!blocks.empty() && !blocks.back().used) {      // grow the free tail block
      Block& b = blocks.back();
      end = b.off + size;
      b.size = size;
      b.used = true;
      return b.off;
    }
    blocks.push_back(Block{end, size, true});
    end += size;
    return blocks.back().off;
  }
  void give(size_t off) {
    for (size_t i = 0; i < blocks.size(); ++i) {
      if (blocks[i].off != off) continue;
      blocks[i].used = false;
      if (i + 1 < blocks.size() && !blocks[i + 1].used) {
        blocks[i].size += blocks[i + 1].size;
        blocks.erase(blocks.begin() + i + 1);
      }
      if (i > 0 && !blocks[i - 1].used) {
        blocks[i - 1].size += blocks[i].size;
        blocks.erase(blocks.begin() + i);
      }
      return;
    }
  }
};

bool nchw(const mg3m_net& n) { return n.layout == MG3M_LAYOUT_NCHW; }

mg3m::ConvGeom conv_geom(const mg3m_net& n, int i) {
  const mg3m_layer& L = n.layers[i];
  const int in = L.input;
  return mg3m::ConvGeom{n.N, n.C[in], n.H[in], n.W[in], L.K, L.R, L.S, L.stride, L.stride,
                        L.pad, L.pad, MG3M_LAYOUT_HWCN, false};
}

// The HWCN tensor layer code reads or writes for activation id: the caller's
// x and y in an HWCN network, arena blocks otherwise.
const float* act_ptr(const mg3m_net& n, int id, const float* x, float* y) {
  if (!nchw(n) && id == 0) return x;
  if (!nchw(n) && id == (int)n.layers.size()) return y;
  return reinterpret_cast<const float*>(n.arena + n.offset[id]);
}

// Infer the shape of every activation from the input's (C0, H0, W0), check
// every layer and plan every convolution.
int build(mg3m_net& n, int C0, int H0, int W0) {
  const int L = (int)n.layers.size();
  n.C.assign(L + 1, 0);
  n.H.assign(L + 1, 0);
  n.W.assign(L + 1, 0);
  n.C[0] = C0;
  n.H[0] = H0;
  n.W[0] = W0;
  n.ws_bytes = 0;
  n.wt_bytes = 0;
  n.wt_off.assign(L, -1);
  for (int i = 0; i < L; ++i) {
    const mg3m_layer& ly = n.layers[i];
    if (ly.input < 0 || ly.input > i) return mg3m::set_error(MG3M_ERR_ARG, at(i) + "input must be an earlier activation");
    const int in = ly.input;
    if (ly.op == MG3M_OP_CONV) {
      if (ly.w == nullptr) return mg3m::set_error(MG3M_ERR_NULL, at(i) + "filter pointer is NULL");
      if (ly.relu != 0 && ly.relu != 1) return mg3m::set_error(MG3M_ERR_ARG, at(i) + "relu must be 0 or 1");
      mg3m::ConvShape s;
      mg3m::Plan p;
      int rc = mg3m::conv_plan(conv_geom(n, i), nullptr, &s, &p);
      if (rc) return mg3m::set_error(rc, at(i) + mg3m_last_error());
      n.C[i + 1] = ly.K;
      n.H[i + 1] = s.Ho;
      n.W[i + 1] = s.Wo;
      n.ws_bytes = std::max(n.ws_bytes, p.ws_bytes);
      if (nchw(n)) {
        n.wt_off[i] = (long long)n.wt_bytes;
        n.wt_bytes += round_up(4 * (size_t)ly.K * n.C[in] * ly.R * ly.S);
      }
      if (ly.add != -1) {
        if (ly.add < 0 || ly.add > i) return mg3m::set_error(MG3M_ERR_ARG, at(i) + "add must be an earlier activation or -1");
        if (n.C[ly.add] != ly.K || n.H[ly.add] != s.Ho || n.W[ly.add] != s.Wo)
          return mg3m::set_error(MG3M_ERR_SHAPE, at(i) + "the added activation's shape differs from the output's");
      }
    } else if (ly.op == MG3M_OP_MAXPOOL) {
      if (ly.add != -1 || ly.relu != 0)
        return mg3m::set_error(MG3M_ERR_ARG, at(i) + "a pooling layer takes no add and no relu");
      std::string err;
      int Ho = 0, Wo = 0;
      int rc = mg3m::maxpool_dims(n.H[in], n.W[in], ly.R, ly.S, ly.stride, ly.stride, ly.pad, ly.pad, &Ho, &Wo, &err);
      if (rc) return mg3m::set_error(rc, at(i) + err);
      n.C[i + 1] = n.C[in];
      n.H[i + 1] = Ho;
      n.W[i + 1] = Wo;
    } else {
      return mg3m::set_error(MG3M_ERR_ARG, at(i) + "unknown op");
    }
    const long long elems = (long long)n.N * n.C[i + 1] * n.H[i + 1] * n.W[i + 1];
    if (elems > mg3m::kMaxTensorBytes / 4)
      return mg3m::set_error(MG3M_ERR_TOO_LARGE, at(i) + "activation larger than 4 GiB - 64 bytes");
  }
  n.ws_bytes = round_up(n.ws_bytes);
  return MG3M_OK;
}

// Offsets of activations 1 .. L-1 (and, in an NCHW network, of the HWCN
// copies of the input, 0, and of the output, L).  keep_all: one block each.
// Otherwise the block of activation j is released after layer last_use[j]
// has run, so it is never handed to a layer that still reads j (a layer's
// output never shares space with its own inputs).
void place(mg3m_net& n, bool keep_all) {
  const int L = (int)n.layers.size();
  std::vector<int> last_use(L + 1, -1);
  for (int i = 0; i < L; ++i) {
    last_use[n.layers[i].input] = i;
    if (n.layers[i].op == MG3M_OP_CONV && n.layers[i].add >= 0) last_use[n.layers[i].add] = i;
  }
  n.offset.assign(L + 1, -1);
  Arena arena;
  auto bytes_of = [&](int id) { return round_up(4 * (size_t)n.N * n.C[id] * n.H[id] * n.W[id]); };
  if (nchw(n)) n.offset[0] = (long long)arena.take(bytes_of(0));
  const int first = nchw(n) ? 0 : 1;        // activations whose block the arena owns
  const int last = nchw(n) ? L : L - 1;
  for (int i = 0; i < L; ++i) {
    const int out = i + 1;
    if (out <= last) n.offset[out] = (long long)arena.take(bytes_of(out));
    if (!keep_all) {
      for (int j = first; j < L; ++j)
        if (last_use[j] == i && n.offset[j] >= 0) arena.give((size_t)n.offset[j]);
    }
  }
  // an activation nobody reads (a dead branch) still gets its own block above
  n.arena_bytes = std::max<size_t>(arena.end, kAlign);
}

int run_layers(mg3m_net& n, const float* x, float* y, hipStream_t stream) {
  const int L = (int)n.layers.size();
  std::string err;
  if (nchw(n)) {
    // the input and every filter to HWCN ([N][C][H][W] -> [H][W][C][N], [K][C][R][S] -> [R][S][C][K])
    int rc = mg3m::launch_swap_outer_inner(x, const_cast<float*>(act_ptr(n, 0, x, y)), n.N, n.C[0],
                                           n.H[0] * n.W[0], stream, &err);
    if (rc == MG3M_OK) rc = mg3m::launch_swap_outer_inner_batch(n.wt_jobs, n.wt_njobs, n.wt_tiles, stream, &err);
    if (rc) return mg3m::set_error(rc, err);
  }
  for (int i = 0; i < L; ++i) {
    const mg3m_layer& ly = n.layers[i];
    const float* src = act_ptr(n, ly.input, x, y);
    float* dst = const_cast<float*>(act_ptr(n, i + 1, x, y));
    const int in = ly.input;
    int rc;
    if (ly.op == MG3M_OP_CONV) {
      const float* add = ly.add >= 0 ? act_ptr(n, ly.add, x, y) : nullptr;
      const float* w = nchw(n) ? n.wt + n.wt_off[i] / 4 : ly.w;
      rc = mg3m::conv_run(src, w, dst, conv_geom(n, i), n.ws, n.ws_bytes, false, nullptr, add, ly.relu,
                          stream);
    } else {
      rc = mg3m::maxpool_run(src, dst, n.N, n.C[in], n.H[in], n.W[in], ly.R, ly.S, ly.stride, ly.stride,
                             ly.pad, ly.pad, MG3M_LAYOUT_HWCN, stream);
    }
    if (rc) return mg3m::set_error(rc, at(i) + mg3m_last_error());
  }
  if (nchw(n)) {
    // the output back to NCHW: [H][W][C][N] -> [N][C][H][W]
    int rc = mg3m::launch_swap_outer_inner(act_ptr(n, L, x, y), y, n.H[L] * n.W[L], n.C[L], n.N, stream, &err);
    if (rc) return mg3m::set_error(rc, err);
  }
  return MG3M_OK;
}

int check_io(const mg3m_net* net, const float* x, float* y) {
  if (net == nullptr || x == nullptr || y == nullptr) return mg3m::set_error(MG3M_ERR_NULL, "net, x and y must be non-NULL");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != net->device)
    return mg3m::set_error(MG3M_ERR_ARG, "the network was created on another device");
  const uintptr_t ax = reinterpret_cast<uintptr_t>(x), ay = reinterpret_cast<uintptr_t>(y);
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(net->arena), a1 = a0 + net->arena_bytes;
  if ((ax >= a0 && ax < a1) || (ay >= a0 && ay < a1))
    return mg3m::set_error(MG3M_ERR_ALIAS, "x or y lies inside the network's arena");
  const uintptr_t f0 = reinterpret_cast<uintptr_t>(net->wt), f1 = f0 + net->wt_bytes;
  if (net->wt != nullptr && ((ax >= f0 && ax < f1) || (ay >= f0 && ay < f1)))
    return mg3m::set_error(MG3M_ERR_ALIAS, "x or y lies inside the network's filter copies");
  return MG3M_OK;
}

void drop_graph(mg3m_net* n) {
  if (n->exec) (void)hipGraphExecDestroy(n->exec);
  if (n->graph) (void)hipGraphDestroy(n->graph);
  n->exec = nullptr;
  n->graph = nullptr;
  n->gx = nullptr;
  n->gy = nullptr;
  n->gs = nullptr;
}

void release(mg3m_net* n) {
  drop_graph(n);
  if (n->arena) (void)hipFree(n->arena);
  if (n->ws) (void)hipFree(n->ws);
  if (n->wt) (void)hipFree(n->wt);
  if (n->wt_jobs) (void)hipFree(n->wt_jobs);
  n->arena = nullptr;
  n->ws = nullptr;
  n->wt = nullptr;
  n->wt_jobs = nullptr;
}

}  // namespace

namespace mg3m {

int prepare_swap_batch(SwapJob* jobs, int n, unsigned* tiles, std::string* err) {
  long long total = 0;
  for (int i = 0; i < n; ++i) {
    SwapJob& j = jobs[i];
    if (j.in == nullptr || j.out == nullptr || j.A < 1 || j.Cm < 1 || j.B < 1) {
      *err = "internal: empty layout change in a batch";
      return MG3M_ERR_SHAPE;
    }
    const long long J = (long long)j.Cm * j.B, tj = (J + 63) / 64, ta = (j.A + 63) / 64;
    if (J > 0x7fffffffLL) {
      *err = "layout change: a dimension exceeds the launch grid";
      return MG3M_ERR_TOO_LARGE;
    }
    j.tiles_j = (unsigned)tj;
    j.tile0 = (unsigned)total;
    j.vl = J % 4 == 0 && (reinterpret_cast<uintptr_t>(j.in) & 15) == 0;
    j.vs = j.A % 4 == 0 && (reinterpret_cast<uintptr_t>(j.out) & 15) == 0;
    total += tj * ta;
    if (total > (1LL << 24) - 1) {
      *err = "layout change: the batch exceeds the launch grid";
      return MG3M_ERR_TOO_LARGE;
    }
  }
  *tiles = (unsigned)total;
  return MG3M_OK;
}

}  // namespace mg3m

extern "C" {

int mg3m_net_create(const mg3m_layer* layers, int n_layers, int N, int C, int H, int W, int layout,
                    int keep_all, mg3m_net** net) {
  mg3m_net* n = nullptr;
  try {
    mg3m::clear_error();
    if (net == nullptr || layers == nullptr) return mg3m::set_error(MG3M_ERR_NULL, "layers and net must be non-NULL");
    *net = nullptr;
    if (n_layers < 1) return mg3m::set_error(MG3M_ERR_ARG, "a network needs at least one layer");
    if (layout != MG3M_LAYOUT_HWCN && layout != MG3M_LAYOUT_NCHW) return mg3m::set_error(MG3M_ERR_LAYOUT, "unknown layout");
    if (N < 1 || C < 1 || H < 1 || W < 1) return mg3m::set_error(MG3M_ERR_SHAPE, "input dimensions must be >= 1");
    if (keep_all != 0 && keep_all != 1) return mg3m::set_error(MG3M_ERR_ARG, "keep_all must be 0 or 1");
    n = new mg3m_net();
    n->layout = layout;
    n->N = N;
    n->layers.assign(layers, layers + n_layers);
    int rc = build(*n, C, H, W);
    if (rc) {
      delete n;
      return rc;
    }
    place(*n, keep_all == 1);
    hipError_t e = hipGetDevice(&n->device);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&n->arena), n->arena_bytes);
    if (e == hipSuccess && n->ws_bytes > 0) e = hipMalloc(&n->ws, n->ws_bytes);
    if (e == hipSuccess && n->wt_bytes > 0) e = hipMalloc(reinterpret_cast<void**>(&n->wt), n->wt_bytes);
    if (e != hipSuccess) {
      release(n);
      delete n;
      return mg3m::set_error(MG3M_ERR_HIP, std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    if (n->wt != nullptr) {
      // the filter copies: [K][C][R*S] -> [R*S][C][K], one job per convolution
      std::vector<mg3m::SwapJob> jobs;
      for (int i = 0; i < n_layers; ++i) {
        const mg3m_layer& ly = n->layers[i];
        if (ly.op != MG3M_OP_CONV) continue;
        mg3m::SwapJob j{};
        j.in = ly.w;
        j.out = n->wt + n->wt_off[i] / 4;
        j.A = ly.K;
        j.Cm = n->C[ly.input];
        j.B = ly.R * ly.S;
        jobs.push_back(j);
      }
      std::string err;
      rc = mg3m::prepare_swap_batch(jobs.data(), (int)jobs.size(), &n->wt_tiles, &err);
      if (rc == MG3M_OK) {
        e = hipMalloc(reinterpret_cast<void**>(&n->wt_jobs), jobs.size() * sizeof(mg3m::SwapJob));
        if (e == hipSuccess)
          e = hipMemcpy(n->wt_jobs, jobs.data(), jobs.size() * sizeof(mg3m::SwapJob), hipMemcpyHostToDevice);
        if (e != hipSuccess) rc = MG3M_ERR_HIP, err = std::string("filter copy table: ") + hipGetErrorString(e);
      }
      if (rc) {
        release(n);
        delete n;
        return mg3m::set_error(rc, err);
      }
      n->wt_njobs = (int)jobs.size();
    }
    *net = n;
    return MG3M_OK;
  } catch (const std::exception& ex) {
    if (n) release(n);
    delete n;
    return mg3m::set_error(MG3M_ERR_HIP, ex.what());
  }
}

int mg3m_net_activation(const mg3m_net* net, int id, int* C, int* H, int* W, const float** ptr) {
  mg3m::clear_error();
  if (net == nullptr || C == nullptr || H == nullptr || W == nullptr)
    return mg3m::set_error(MG3M_ERR_NULL, "net, C, H and W must be non-NULL");
  const int L = (int)net->layers.size();
  if (id < 0 || id > L) return mg3m::set_error(MG3M_ERR_ARG, "activation id out of range");
  *C = net->C[id];
  *H = net->H[id];
  *W = net->W[id];
  if (ptr) *ptr = (id == 0 || id == L) ? nullptr : reinterpret_cast<const float*>(net->arena + net->offset[id]);
  // (stored activations are HWCN in every network)
  return MG3M_OK;
}

int mg3m_net_memory(const mg3m_net* net, size_t* arena_bytes, size_t* workspace_bytes) {
  mg3m::clear_error();
  if (net == nullptr || arena_bytes == nullptr || workspace_bytes == nullptr)
    return mg3m::set_error(MG3M_ERR_NULL, "net and out-parameters must be non-NULL");
  *arena_bytes = net->arena_bytes;
  *workspace_bytes = net->ws_bytes + net->wt_bytes;
  return MG3M_OK;
}

int mg3m_net_forward(mg3m_net* net, const float* x, float* y, void* stream) {
  try {
    mg3m::clear_error();
    int rc = check_io(net, x, y);
    if (rc) return rc;
    return run_layers(*net, x, y, static_cast<hipStream_t>(stream));
  } catch (const std::exception& e) {
    return mg3m::set_error(MG3M_ERR_HIP, e.what());
  }
}

int mg3m_net_forward_graph(mg3m_net* net, const float* x, float* y, void* stream) {
  try {
    mg3m::clear_error();
    int rc = check_io(net, x, y);
    if (rc) return rc;
    if (stream == nullptr) return mg3m::set_error(MG3M_ERR_ARG, "graph capture needs a non-default stream");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (net->exec == nullptr || net->gx != x || net->gy != y || net->gs != s) {
      drop_graph(net);
      hipError_t e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
      if (e != hipSuccess) return mg3m::set_error(MG3M_ERR_HIP, std::string("hipStreamBeginCapture: ") + hipGetErrorString(e));
      rc = run_layers(*net, x, y, s);
      hipGraph_t g = nullptr;
      e = hipStreamEndCapture(s, &g);
      if (rc) {
        if (g) (void)hipGraphDestroy(g);
        return rc;
      }
      if (e != hipSuccess) return mg3m::set_error(MG3M_ERR_HIP, std::string("hipStreamEndCapture: ") + hipGetErrorString(e));
      net->graph = g;
      e = hipGraphInstantiate(&net->exec, g, nullptr, nullptr, 0);
      if (e != hipSuccess) {
        drop_graph(net);
        return mg3m::set_error(MG3M_ERR_HIP, std::string("hipGraphInstantiate: ") + hipGetErrorString(e));
      }
      net->gx = x;
      net->gy = y;
      net->gs = s;
    }
    hipError_t e = hipGraphLaunch(net->exec, s);
    if (e != hipSuccess) return mg3m::set_error(MG3M_ERR_HIP, std::string("hipGraphLaunch: ") + hipGetErrorString(e));
    return MG3M_OK;
  } catch (const std::exception& e) {
    return mg3m::set_error(MG3M_ERR_HIP, e.what());
  }
}

int mg3m_net_destroy(mg3m_net* net) {
  mg3m::clear_error();
  if (net == nullptr) return MG3M_OK;
  release(net);
  delete net;
  return MG3M_OK;
}

}  // extern "C"
