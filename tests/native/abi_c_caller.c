/* A plain C99 caller of the library (no GPU needed): the header compiles as
   C, the exported symbols link, and host-side validation answers before any
   device work. */
#include <stdio.h>
#include <string.h>
#include "fork_step.h"
int main(void) {
  fork_step_args a;
  memset(&a, 0, sizeof a);
  if (fork_version() != 10100) return 1;
  if (fork_step_ex(NULL) != FORK_EINVAL) return 2;
  if (strlen(fork_last_error()) == 0) return 3;
  a.B = 2; a.L = 8; a.d = 16; a.V = 100; a.block_len = 4; a.tau = 0.9f;
  if (fork_step_ex(&a) != FORK_EINVAL) return 4; /* NULL arrays */
  if (fork_workspace_bytes(8, 512, 126464) == 0) return 5;
  printf("c abi ok: %s\n", fork_last_error());
  return 0;
}
