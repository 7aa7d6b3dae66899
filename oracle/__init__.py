"""Plain float64 CPU oracle for the D^2SD verify step (arXiv 2606.04446).

TEST INFRASTRUCTURE, NOT PRODUCT CODE. Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import it. It shares no code with the HIP
path (``paper_2606_04446_amd``) and imports nothing from it.

Each function computes the plain definition of its step, slowly and visibly:

  tree       candidate tree from (B, p_k): sec. 3.2 (branch construction after
             Eq. 5) and sec. 3.3 (ii)-(iii); ancestor sets by walking parents
  attention  softmax attention of every tree node over the context plus its
             ancestors-or-self (sec. 3.3 (iv), shared-prefix joint
             verification), and the log-sum-exp merge of two states
  accept     longest accepted prefix across the candidate paths and the bonus
             token (sec. 2 "DFlash", sec. 3.3 (iv)), two independent ways
  boundary   rejection-boundary posterior r(i) (Eq. 4) and top-K prefix
             lengths (Eq. 5)
  commit     the accepted path's K/V appended to the paged context (sec. 3.3:
             each cycle consumes the verified cache and the bonus anchor)
  sampling   verification at T > 0 (Tables 3-4 report T = 1; the tree rule is
             a reading): one target draw per distinct context by inversion,
             then the greedy longest-path rule on the drawn tokens

Readings of points the paper leaves open are listed with each function.
"""
