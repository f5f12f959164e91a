/* Allocation-failure injection for the host-robustness test: preloaded
 * (LD_PRELOAD) in a child process, it makes every malloc-family request of
 * at least `limit` bytes fail once failalloc_arm(limit) is called (operator
 * new then throws std::bad_alloc). Test infrastructure only. */
#define _GNU_SOURCE
#include <errno.h>
#include <stddef.h>

extern void* __libc_malloc(size_t);
extern void* __libc_calloc(size_t, size_t);
extern void* __libc_realloc(void*, size_t);
extern void* __libc_memalign(size_t, size_t);

static volatile size_t g_limit = 0; /* 0: disarmed */
static volatile long g_refused = 0;

void failalloc_arm(size_t limit) {
  g_limit = limit;
  g_refused = 0;
}
long failalloc_refused(void) { return g_refused; }

static int refuse(size_t n) {
  if (g_limit != 0 && n >= g_limit) {
    ++g_refused;
    errno = ENOMEM;
    return 1;
  }
  return 0;
}

void* malloc(size_t n) { return refuse(n) ? NULL : __libc_malloc(n); }
void* calloc(size_t a, size_t b) { return refuse(a * b) ? NULL : __libc_calloc(a, b); }
void* realloc(void* p, size_t n) { return refuse(n) ? NULL : __libc_realloc(p, n); }
void* memalign(size_t al, size_t n) { return refuse(n) ? NULL : __libc_memalign(al, n); }
void* aligned_alloc(size_t al, size_t n) { return refuse(n) ? NULL : __libc_memalign(al, n); }
int posix_memalign(void** p, size_t al, size_t n) {
  if (refuse(n)) return ENOMEM;
  void* q = __libc_memalign(al, n);
  if (q == NULL) return ENOMEM;
  *p = q;
  return 0;
}
