"""CPU oracle for speculative rejection-sampling verification and the TV loss.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 restatement
of what the paper ("Breaking Entropy Bounds: Accelerating RL Training via MTP
with Rejection Sampling") defines.  It exists so that the GPU path can be
checked against something written independently of it.  Only the test suite,
the smoke check of ``__graft_entry__`` and the CPU-baseline leg of
``bench.py`` may import it; the library itself never does, and it shares no
code, header, table or constant generator with the HIP sources.

Modules
-------
philox   Philox4x64-10 counter-based generator (Salmon et al., SC'11).
verify   Chain rejection-sampling verification (Sec. 2.2 Eq. reject_sample,
         App. G.1 Alg. rs_multinomial).
tv       TV loss, its gradient and the end-to-end multi-step TV loss
         (Sec. 4.1 Eqs. tv_loss / tv_grad, Sec. 4.2 Eq. e2e_tv, App. A).
variants Target-only verification (Sec. 2.2 Eq. target_only), the draft-stage
         sampler (App. G.1 draft stage) and per-step diagnostics (entropies,
         alpha^TO, alpha^RS and its split, the App. E decision boundary).
gumbel   Gumbel-max verification (App. G.2, Alg. rs_gumbel) and the
         Gumbel-max draft sampler.
kl       CE, forward-KL and reverse-KL losses and gradients (Sec. 4.1 and its
         footnote, Table grad_comparison, App. B, App. C).

Every function is pinned by the ``-m "not gpu"`` tests against something
other than itself (numpy's own Philox, scipy routines, closed forms,
invariants, brute force, finite differences, chi-square statistics).
"""

from .philox import philox4x64_10, u24, draw_words  # noqa: F401
from .verify import verify_ref, softmax_t, residual_sample  # noqa: F401
from .tv import tv_ref, chain_factors  # noqa: F401
