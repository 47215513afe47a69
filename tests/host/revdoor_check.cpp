#include "../../paper_2608_25230_amd/csrc/revdoor.hpp"
#include <cstdio>
#include <set>
#include <vector>
#include <cstdint>
int main(){
  for (int n=1;n<=14;++n) for (int t=0;t<=n;++t){
    int c[70]; fw::revdoor_init(c,t,n);
    std::set<uint64_t> seen; std::vector<uint64_t> seq;
    auto mask=[&](){uint64_t m=0; for(int j=1;j<=t;++j) m|=1ull<<c[j]; return m;};
    uint64_t m=mask(); seen.insert(m); seq.push_back(m);
    int in,out;
    while(fw::revdoor_next(c,t,&in,&out)){
      uint64_t m2=mask();
      if (m2 != ((m ^ (1ull<<in)) ^ (1ull<<out)) || !(m>>out&1) || (m>>in&1)) {printf("bad step n=%d t=%d\n",n,t); return 1;}
      for(int j=1;j<t;++j) if(c[j]>=c[j+1]) {printf("unsorted\n");return 1;}
      if(seen.count(m2)){printf("dup n=%d t=%d\n",n,t);return 1;}
      seen.insert(m2); seq.push_back(m2); m=m2;
    }
    // count
    double C=1; for(int i=1;i<=t;++i) C=C*(n-t+i)/i;
    if ((double)seq.size()!= C){printf("count n=%d t=%d got %zu want %.0f\n",n,t,seq.size(),C);return 1;}
    // unranking gives every position of the walk
    for(size_t i=0;i<seq.size();++i) if (fw::revdoor_unrank(i,n,t)!=seq[i]) {printf("unrank n=%d t=%d r=%zu\n",n,t,i);return 1;}
    // prefix property
    for(int b=t;b<=n;++b){ double Cb=1; for(int i=1;i<=t;++i) Cb=Cb*(b-t+i)/i;
      for(size_t i=0;i<(size_t)Cb;++i) if (seq[i]>>b) {printf("prefix n=%d t=%d b=%d\n",n,t,b);return 1;} }
  }
  printf("revolving door OK\n"); return 0;
}
