// Trace of the executor's stream operations recorded by trace_stubs.cpp.
#pragma once
#include <cstdint>
#include <vector>

// Byte range [lo, hi) of device memory a launch reads or writes.
struct Span {
  uintptr_t lo, hi;
  bool write;
};
struct TraceOp {
  char kind;         // 'K' launch, 'R' event record, 'W' stream waits for an event
  uintptr_t stream;  // stream handle
  uintptr_t event;   // event handle ('R', 'W')
  const char *what;
  bool known;        // 'K': the spans below are the launch's whole footprint
  std::vector<Span> spans;
};
extern std::vector<TraceOp> g_trace;
