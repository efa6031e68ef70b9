// Graph capture of the library's calls (GRACE captures its whole fixed-length
// decoding loop as one graph, Sec. 5): every entry point only enqueues kernels
// on the caller's stream and never allocates, synchronises or sets memory, so
// a decode loop recorded between grace_graph_begin and grace_graph_end replays
// with one launch.
#include <hip/hip_runtime.h>

#include "../../include/grace.h"

namespace {
thread_local int32_t g_graph_error = 0;

int32_t graph_status(hipError_t e) {
  if (e == hipSuccess) return GRACE_OK;
  g_graph_error = (int32_t)e;
  return GRACE_ERR_HIP;
}
}  // namespace

extern "C" {

int32_t grace_graph_begin(void* stream) {
  if (stream == nullptr) return GRACE_ERR_NULL;   // the null stream cannot be captured
  return graph_status(hipStreamBeginCapture((hipStream_t)stream, hipStreamCaptureModeThreadLocal));
}

int32_t grace_graph_end(void* stream, void** graph_exec) {
  if (stream == nullptr || graph_exec == nullptr) return GRACE_ERR_NULL;
  *graph_exec = nullptr;
  hipGraph_t graph = nullptr;
  hipError_t e = hipStreamEndCapture((hipStream_t)stream, &graph);
  if (e != hipSuccess) return graph_status(e);
  hipGraphExec_t exec = nullptr;
  e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  const hipError_t e2 = hipGraphDestroy(graph);
  if (e != hipSuccess) return graph_status(e);
  if (e2 != hipSuccess) {
    (void)hipGraphExecDestroy(exec);
    return graph_status(e2);
  }
  *graph_exec = (void*)exec;
  return GRACE_OK;
}

int32_t grace_graph_launch(void* graph_exec, void* stream) {
  if (graph_exec == nullptr) return GRACE_ERR_NULL;
  return graph_status(hipGraphLaunch((hipGraphExec_t)graph_exec, (hipStream_t)stream));
}

int32_t grace_graph_destroy(void* graph_exec) {
  if (graph_exec == nullptr) return GRACE_OK;
  return graph_status(hipGraphExecDestroy((hipGraphExec_t)graph_exec));
}

int32_t grace_graph_last_hip_error(void) { return g_graph_error; }

}  // extern "C"
