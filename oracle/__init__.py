"""CPU oracle for the DBLast head and stochastic-verification hot path.

TEST INFRASTRUCTURE, not part of the product. Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import, call or execute anything in this package; the
HIP library and its Python binding never do, and this package imports nothing from them.

It is a plain, slow restatement of what the paper defines, in binary64 unless the
determinism contract (``oracle/contract.py``) fixes another precision for a discrete decision:

* ``oracle.contract``  Philox4x32-10 draws, deterministic exponentials, 2^-40 quantisation,
                       integer inverse CDF and accept test;
* ``oracle.head``      the output head: logits through the shared LM head, log-softmax over V,
                       and its two-level (tile) form;
* ``oracle.mixture``   category prior, block draw, category posterior, sequential accept test,
                       residual and bonus draws, acceptance mass, AL_b and expected length;
* ``oracle.enumerate`` exact expected accepted length by enumerating every block (tiny V, K).
"""
from . import contract, enumerate, head, mixture  # noqa: F401
