"""Plain, slow, fp64 CPU oracle for the packed-MLP training step.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this package: only the test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, tables or
constants with the HIP library; the only thing both sides consume in common is
the seeded synthetic data produced by ``paper_2607_05380_amd.synth`` (which
holds none of the method's arithmetic).

What it computes (arXiv 2607.05380, "TabPack"):

* §3.3 Model Pack -- a pack of m MLPs built from Linear-ReLU-Dropout blocks,
  each member with its own width and dropout rate, must behave exactly like
  the m separate MLPs.  The oracle therefore *is* m separate MLPs, one Python
  loop iteration per member, in numpy float64.
* §3.4 Optimizer Pack -- one optimizer per member with its own learning rate
  and weight decay (AdamW here, see ``mlp.adamw_step``).
* §3.6 Training -- each member sees its own base batch; the members' losses
  are summed, never their predictions.
* §3.5 Ensemble -- greedy ensembling over a candidate pool (``greedy``), and
  the online ensemble rebuilt every epoch from the members' latest states and
  the previous ensemble, with early stopping of base models and of the
  ensemble (§3.6) (``online``).
* §3.7 / App. F hyperparameter space -- members' hyperparameters are drawn
  from ranges (``sampling``).

Modules
-------
philox    Philox4x32-10 / Philox4x64-10 block functions (Salmon et al., SC'11).
sampling  hyperparameter draws and nn.Linear-style initial parameters.
mlp       one member: forward, loss, backward, AdamW, dropout masks.
pack      K independent members: one training step, evaluation, scores.
greedy    greedy ensemble selection.
online    the per-epoch online loop: validation, member removal, ensemble
          rebuild, early stopping, the final ensemble's prediction.

Parity pins (tests/test_oracle_*.py) tie every function to something other
than itself: published Philox known-answer vectors and numpy's Philox,
central finite differences, torch float64 autograd, torch.optim.AdamW,
closed forms, brute-force greedy search, a hand-worked greedy example, a
hand-worked online run and closed forms of the online loop's stopping rules.
"""
