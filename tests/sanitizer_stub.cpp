// Host-only stand-in for the error-message functions of libparrot_attn, so
// that context_store.cpp can be built alone with g++ under AddressSanitizer
// and UndefinedBehaviorSanitizer (tests/test_store_sanitized.py).
#include <cstdarg>
#include <cstdio>
#include <string>
#include "parrot_attn.h"
namespace parrot {
static thread_local std::string g_msg;
parrot_status set_error(parrot_status s, const char* fmt, ...) {
  if (s == PARROT_OK) { g_msg.clear(); return s; }
  char buf[512]; va_list ap; va_start(ap, fmt); vsnprintf(buf, sizeof buf, fmt, ap); va_end(ap);
  g_msg = buf; return s;
}
}
extern "C" const char* parrot_last_error(void) { return parrot::g_msg.c_str(); }
