/* The C ABI from plain C11: the header compiles with -std=c11 -pedantic as C
 * (not C++), and a C program links against liboptimus.so and calls its
 * host-only entry points. Descriptors name addresses only; validation never
 * dereferences them, so none is allocated. Prints "ok" on success. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "optimus.h"

static int check(const char* what, optimus_status got, optimus_status want) {
  if (got != want) {
    printf("%s: status %d, expected %d (%s)\n", what, (int)got, (int)want, optimus_last_error());
    return 1;
  }
  return 0;
}

int main(void) {
  int bad = 0;
  const char* v = optimus_version();
  if (!v || !*v) {
    printf("empty version\n");
    return 1;
  }
  /* two bf16 members, 16-byte aligned addresses, outputs apart from inputs */
  optimus_linear_desc d[2];
  memset(d, 0, sizeof d);
  d[0].x = (const void*)(uintptr_t)0x100000; d[0].ldx = 64;
  d[0].w = (const void*)(uintptr_t)0x200000; d[0].ldw = 64;
  d[0].bias = (const void*)(uintptr_t)0x300000;
  d[0].y = (void*)(uintptr_t)0x400000; d[0].ldy = 32;
  d[0].M = 100; d[0].N = 32; d[0].K = 64;
  d[1] = d[0];
  d[1].y = (void*)(uintptr_t)0x500000;
  d[1].M = 7;
  bad |= check("valid group", optimus_validate_linear(d, 2, OPTIMUS_BF16, OPTIMUS_ACT_SIGMOID), OPTIMUS_OK);
  bad |= check("empty group", optimus_validate_linear(d, 0, OPTIMUS_BF16, OPTIMUS_ACT_NONE), OPTIMUS_OK);
  /* a row stride shorter than the row */
  optimus_linear_desc e = d[0];
  e.ldx = 16;
  bad |= check("short ldx", optimus_validate_linear(&e, 1, OPTIMUS_BF16, OPTIMUS_ACT_NONE), OPTIMUS_ERR_INVALID_ARG);
  /* the second member's output is the first member's input */
  optimus_linear_desc a[2] = {d[0], d[1]};
  a[1].y = (void*)(uintptr_t)0x100000;
  a[1].ldy = 64;
  bad |= check("aliasing", optimus_validate_linear(a, 2, OPTIMUS_BF16, OPTIMUS_ACT_NONE), OPTIMUS_ERR_ALIASING);
  /* an unknown activation value (the header: OPTIMUS_ERR_UNSUPPORTED) */
  bad |= check("unknown act", optimus_validate_linear(d, 2, OPTIMUS_BF16, (optimus_act)99), OPTIMUS_ERR_UNSUPPORTED);
  if (!optimus_last_error() || !*optimus_last_error()) {
    printf("no error text after a failed validation\n");
    bad = 1;
  }
  if (!bad) printf("ok %s\n", v);
  return bad;
}
