"""Generation-state signals of the trajectory risk (Sec. 4.2, before Eq. 7).

After step t: c_t is the mean confidence of the provisional predictions over
the answer positions still unresolved, and chi_t is the fraction of the
positions unresolved at both steps t-1 and t whose highest-logit token
changed between the two updates (chi_1 = 0).  Reading: "unresolved" is the
set still masked after the step-t commitment (M_{t+1}); an empty set gives
c = 0 and chi = 0.  Sums run in ascending position order in double.
"""


def mean_conf(conf, masked_after) -> float:
    s = 0.0
    n = 0
    for i in range(len(masked_after)):
        if masked_after[i]:
            s = s + float(conf[i])
            n += 1
    return 0.0 if n == 0 else s / n


def churn(argmax_now, argmax_prev, masked_after, first_step: bool) -> float:
    if first_step:
        return 0.0
    n = 0
    ch = 0
    for i in range(len(masked_after)):
        if masked_after[i]:
            n += 1
            if int(argmax_now[i]) != int(argmax_prev[i]):
                ch += 1
    return 0.0 if n == 0 else ch / n
